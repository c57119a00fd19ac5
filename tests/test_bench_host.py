"""Host logic of bench.py: the one-GPU guard, the algorithmic byte and flop
counts against their closed forms, the roofline classification, the choice
of the dominant kernel and the lookup of the committed counter figures.
None of it touches a GPU."""

import json
import os
import subprocess
import sys
import types

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2608_25332_amd import workloads as W  # noqa: E402

LARGE = [2, 3, 4, 5]


def fake_workload(wid):
    """What algorithmic() and rooflines() read of a workload, without drawing
    its tensors."""
    s = W.WORKLOADS[wid]
    return types.SimpleNamespace(spec=s, N1=s.N1, N2=s.N2, dtype=s.dtype,
                                 heads=np.zeros((s.B, s.n_heads), np.int32))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"] and msg["gpus_requested"] == 2


@pytest.mark.parametrize("wid", LARGE)
def test_algorithmic_closed_forms(wid):
    w = fake_workload(wid)
    s = w.spec
    e = 2 if s.dtype == "bf16" else 4
    kern, stage = bench.algorithmic(w)
    Mp = s.Nv - s.N1
    # the Gram multiplies every pruned row with every kept row over d
    assert kern["gram_tile"]["flops"] == 2.0 * s.B * Mp * s.N1 * s.d
    assert kern["gram_tile"]["bytes"] == s.B * s.Nv * s.d * e
    # the merge reads every visual row and writes the N1 centroids
    assert kern["merge"]["bytes"] == s.B * (s.Nv + s.N1) * s.d * e
    # the score touches the selected heads only
    assert kern["score_partial"]["bytes"] == s.B * s.n_heads * (s.Nt + s.N1) * s.hd * e
    # every kernel belongs to a stage the stage table prices
    assert set(bench.STAGE_OF) <= set(kern)
    assert set(bench.STAGE_OF.values()) == set(stage)
    # a shared launch does the work of its parts (the merge writes the kept
    # rows in place, so its compaction reads no merged row)
    for name, parts in bench.SHARED_PARTS.items():
        fl = sum(kern[p]["flops"] for p in parts)
        by = sum(kern[p]["bytes"] for p in parts)
        if name == "merge+gather_hkv2":
            by -= s.B * s.N2 * s.d * e
        assert kern[name]["flops"] == fl and kern[name]["bytes"] == by
    for v in list(kern.values()) + list(stage.values()):
        assert v["bytes"] > 0 and v["flops"] >= 0


def test_roof_bound_and_units():
    ridge = bench.BF16_PEAK_TFLOPS * 1e12 / (bench.HBM_PEAK_GBS * 1e9)
    # 1 GB in 1 ms is 1000 GB/s, an eighth of the HBM peak
    r = bench.roof({"bytes": 1e9, "flops": 0.0}, 1e-3)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s"
    assert r["achieved"] == pytest.approx(1000.0) and r["frac"] == pytest.approx(0.125)
    # above the ridge the same bytes are priced against the matrix cores
    r = bench.roof({"bytes": 1e9, "flops": 2 * ridge * 1e9}, 1e-3)
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s"
    assert r["frac"] == pytest.approx(r["achieved"] / bench.BF16_PEAK_TFLOPS)
    # the large Grams are above the ridge, the merge and the compaction below
    for wid in (4, 5):
        kern, _ = bench.algorithmic(fake_workload(wid))
        assert bench.roof(kern["gram_tile"], 1e-5)["bound"] == "mfma"
        assert bench.roof(kern["merge"], 1e-5)["bound"] == "hbm"
        assert bench.roof(kern["gather_hkv2"], 1e-5)["bound"] == "hbm"


def test_dominant_kernel_and_traffic(monkeypatch):
    w = fake_workload(4)
    seen = []

    def traffic(name, kernel):
        seen.append((name, kernel))
        return 123.0

    monkeypatch.setattr(bench, "load_traffic", traffic)
    kern_us = {"cos_partial": 10.0, "gram_tile": 60.0, "merge": 20.0, "select": 3.0}
    rf, kernels, stages, shared, stage_us = bench.rooflines(w, "one_stream", kern_us, {})
    assert rf["kernel"] == "gram_tile" and rf["kernel_us"] == 60.0
    assert rf["traffic"] == 123.0 and seen == [(w.spec.name, "gram_tile")]
    assert stage_us == {"cosine": 10.0, "gram": 60.0, "merge": 20.0, "select": 3.0}
    assert "frac_of_bf16_mfma_peak" in kernels["gram_tile"]
    # the shared-launch form takes its dominant kernel among the shared launches
    shared_us = {"gram_partial+score_partial": 5.0, "merge+gather_hkv2": 8.0}
    rf, *_ = bench.rooflines(fake_workload(2), "shared_launches", {"select": 1.0}, shared_us)
    assert rf["kernel"] == "merge+gather_hkv2"


def committed_pmc():
    out = []
    for f in sorted(os.listdir(os.path.join(ROOT, "profiles"))):
        if f.startswith("pmc_") and f.endswith(".md"):
            txt = open(os.path.join(ROOT, "profiles", f)).read()
            i = txt.find("```json")
            j = txt.find("```", i + 7)
            out.append(json.loads(txt[i + 7:j]))
    return out


def test_traffic_lookup(monkeypatch):
    recs = committed_pmc()
    assert {r["workload"] for r in recs} >= {W.WORKLOADS[2].name, W.WORKLOADS[5].name}
    for rec in recs:
        monkeypatch.setattr(bench, "csrc_digest", lambda d=rec["csrc_digest"]: d)
        found = 0
        for kernel in bench.STAGE_OF:
            t = bench.load_traffic(rec["workload"], kernel)
            if t is not None:
                assert np.isfinite(t) and t > 0
                found += 1
        for kernel in bench.SHARED_PARTS:
            t = bench.load_traffic(rec["workload"], kernel)
            assert t is None or t > 0
        assert found >= 4, rec["workload"]
        # figures taken from other sources are not used
        monkeypatch.setattr(bench, "csrc_digest", lambda: "0" * 16)
        assert all(bench.load_traffic(rec["workload"], k) is None for k in bench.STAGE_OF)
    assert bench.load_traffic("no-such-workload", "gram_tile") is None


def test_csrc_digest_is_stable():
    a = bench.csrc_digest()
    assert a == bench.csrc_digest() and len(a) == 16 and int(a, 16) >= 0
