"""Mutation check of the oracle's pins (CPU only).

Each case copies the oracle source, plants one plausible mistake (a dropped
term, a wrong sign, index or axis, a transposed operand), compiles the copy
and runs every pin against it.  At least one pin must fail, otherwise the
pins would not notice that mistake in the oracle.  The mistakes are planted
in the CPU oracle only; every mutant keeps its memory accesses in bounds.
"""
import os
import shutil
import subprocess
import tempfile

import pytest

import oracle
import oracle_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "provip_oracle.c")

# (name, text in the oracle, replacement)
MUTANTS = [
    ("cosine-drop-vis-norm", "double den = tn * sqrt(vv);", "double den = tn;"),
    ("cosine-transposed-out", "M[(size_t)i * nv + j] = (den == 0.0)", "M[(size_t)j * nt + i] = (den == 0.0)"),
    ("cosine-self-dot", "tv += t[c] * v[c];", "tv += v[c] * v[c];"),
    ("center-wrong-count", "double mean = s / (double)nv;", "double mean = s / (double)nt;"),
    ("center-wrong-sign", "M[(size_t)i * nv + j] - mean;", "M[(size_t)i * nv + j] + mean;"),
    ("center-column-mean", "for (int k = 0; k < nv; ++k) s += M[(size_t)i * nv + k];",
     "for (int k = 0; k < nt; ++k) s += M[(size_t)k * nv + (i % nv)];"),
    ("maxpool-min", "if (x > m) m = x;", "if (x < m) m = x;"),
    ("topk-tie-high-index", "(score[jj] == score[j] && jj < j)", "(score[jj] == score[j] && jj > j)"),
    ("topk-ascending", "if (score[jj] > score[j] ||", "if (score[jj] < score[j] ||"),
    ("assign-drop-centroid-norm", "double den = sqrt(xx) * sqrt(yy);", "double den = sqrt(xx);"),
    ("assign-index-not-slot", "bs = s;\n", "bs = kept[s];\n"),
    ("assign-argmin", "if (cs > b) {", "if (bs < 0 || cs < b) {"),
    ("assign-tie-high-slot", "if (cs > b) {", "if (cs >= b) {"),
    ("merge-sum-not-mean", "out[c] /= (double)count;", "out[c] /= 1.0;"),
    ("merge-skip-self", "int count = 1;", "int count = 1; for (int c = 0; c < d; ++c) out[c] = 0.0;"),
    ("attention-scale-hd", "double scale = 1.0 / sqrt((double)hd);", "double scale = 1.0 / (double)hd;"),
    ("attention-no-normalise", "for (int j = 0; j < n; ++j) row[j] /= z;", "(void)z;"),
    ("attention-no-scale", "row[j] = s * scale;", "row[j] = s;"),
    ("headaware-list-position", "k + (size_t)h * n * hd, nt, n, hd, A);", "k + (size_t)t * n * hd, nt, n, hd, A);"),
    ("headaware-mean-over-all-heads", "S[e] /= (double)nh;", "S[e] /= (double)H;"),
    ("headaware-no-row-mean", "v[j] = s / (double)nt;", "v[j] = s;"),
    ("headaware-row-sum-not-col", "for (int i = 0; i < nt; ++i) s += S[(size_t)i * n + j];",
     "for (int i = 0; i < nt; ++i) s += S[(size_t)(j % nt) * n + (i % n)];"),
    ("gather-src-stride", "src + b * sb + g * sg + j * sr", "src + b * sb + j * sr"),
    ("in-model-lse-dropped", "double z = exp(lse[i] - m);", "double z = 0.0;"),
    ("in-model-lse-unshifted", "double z = exp(lse[i] - m);", "double z = exp(lse[i]);"),
    ("in-model-lse-scaled-again", "double z = exp(lse[i] - m);", "double z = exp(lse[i] * scale - m);"),
    ("text-scaled-logits", "row[j] = s;\n        }\n        double m = row[0];\n        for (int j = 1; j < nt; ++j)",
     "row[j] = s / sqrt((double)d);\n        }\n        double m = row[0];\n        for (int j = 1; j < nt; ++j)"),
    ("text-row-mean-not-column", "for (int i = 0; i < nt; ++i) s += S[(size_t)i * nt + j];",
     "for (int i = 0; i < nt; ++i) s += S[(size_t)j * nt + i];"),
    ("text-at-or-above-mean", "mask[j] = r[j] > mean ? 1 : 0;", "mask[j] = r[j] >= mean ? 1 : 0;"),
    ("text-below-mean", "mask[j] = r[j] > mean ? 1 : 0;", "mask[j] = r[j] < mean ? 1 : 0;"),
    ("text-no-fallback", "if (count == 0) {", "if (count < 0) {"),
    ("confidence-no-mean-subtraction", "var += (row[j] - mean) * (row[j] - mean);",
     "var += row[j] * row[j];"),
    ("confidence-sample-variance", "c += var / (double)n;", "c += var / (double)(n - 1);"),
    ("confidence-row-mean-not-sum", "conf[h] = c;", "conf[h] = c / (double)nt;"),
    ("confidence-std-not-var", "c += var / (double)n;", "c += sqrt(var / (double)n);"),
    ("confidence-first-row-only", "for (int i = 0; i < nt; ++i) {\n            const double *row = A + (size_t)i * n;",
     "for (int i = 0; i < 1; ++i) {\n            const double *row = A + (size_t)i * n;"),
    ("visual-heads-lowest", "if (rc == 0) rc = orc_topk(c, H, n_vis, heads);",
     "for (int h = 0; h < H; ++h) c[h] = -c[h];\n    if (rc == 0) rc = orc_topk(c, H, n_vis, heads);"),
    ("confidence-in-model-visual-only",
     "orc_attention_in_model(q + (size_t)h * nt * hd, k + (size_t)h * n * hd,\n                               lse + (size_t)h * nt, nt, n, hd, slice_map);",
     "orc_attention(q + (size_t)h * nt * hd, k + (size_t)h * n * hd, nt, n, hd, slice_map);"),
    ("confidence-in-model-lse-of-head-0", "lse + (size_t)h * nt, nt, n, hd, slice_map);",
     "lse, nt, n, hd, slice_map);"),
    ("confidence-in-model-mean-assumes-unit-mass", "avg /= (double)n;", "avg = 1.0 / (double)n;"),
    ("confidence-in-model-sample-variance", "total += sq_dev / (double)n;",
     "total += sq_dev / (double)(n - 1);"),
    ("confidence-in-model-first-row-only", "const double *slice = slice_map + (size_t)i * n;",
     "const double *slice = slice_map;"),
    ("visual-heads-in-model-lowest", "if (rc == 0) rc = orc_topk(cm, H, n_vis, heads);",
     "for (int h = 0; h < H; ++h) cm[h] = -cm[h];\n    if (rc == 0) rc = orc_topk(cm, H, n_vis, heads);"),
]


@pytest.fixture(scope="module")
def workdir():
    d = tempfile.mkdtemp(prefix="orc_mut_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


def test_mutant_list_applies():
    src = open(SRC).read()
    for name, old, new in MUTANTS:
        assert src.count(old) >= 1, name


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(name, old, new, workdir):
    src = open(SRC).read()
    assert old in src
    msrc = os.path.join(workdir, f"{name}.c")
    with open(msrc, "w") as f:
        f.write(src.replace(old, new, 1))
    lib_path = os.path.join(workdir, f"lib{name}.so")
    oracle.build(lib_path, msrc)
    lib = oracle.load(lib_path)
    failed = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(lib)
        except (AssertionError, oracle.OracleError, ValueError, IndexError):
            failed.append(pin.__name__)
    assert failed, f"no pin catches mutant {name}"
