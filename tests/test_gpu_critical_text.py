"""Critical text tokens (Sec. 4.2) on the GPU against the CPU oracle, and the
two calls that take its mask: pruning before the LLM with the anchors
restricted to the critical rows, and visual-head identification summed over
them.  All calls go through the C ABI."""

from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
from paper_2608_25332_amd import workloads as W
from parity_util import TAU, TOL, check_kept, rel_err, to_dev, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_25332_amd import provip
    provip.load()


def run_text(text_np, dtype):
    from paper_2608_25332_amd import provip
    r = provip.pv_critical_text(to_dev(text_np, dtype))
    torch.cuda.synchronize()
    return to_host(r["mask"]), to_host(r["count"]), to_host(r["r"])


def check_mask(mask, count, r_ref, mask_ref, dtype):
    """The critical set must equal the oracle's except tokens whose oracle r
    lies within TAU of the mean (those may go either way)."""
    for b in range(r_ref.shape[0]):
        assert count[b] == mask[b].sum()
        if mask_ref[b].all() and mask[b].all():
            continue
        mean = r_ref[b].mean()
        tau = TAU[dtype] * np.abs(r_ref[b]).max()
        sure = np.abs(r_ref[b] - mean) > tau
        assert np.array_equal(mask[b][sure], mask_ref[b][sure]), b


TEXT_CASES = [
    # (B, Nt, d, scale, dtype): scale sets how peaked the softmax rows are
    (1, 16, 256, 0.108, "f32"),
    (3, 64, 4096, 0.027, "bf16"),
    (2, 128, 4096, 0.027, "bf16"),
    (4, 37, 1024, 0.054, "bf16"),
    (1, 300, 512, 0.077, "f32"),
    (1, 700, 256, 0.1, "f32"),       # 11 row elements per lane; wide self-similarity tiles
    (2, 1024, 128, 0.15, "bf16"),    # the most text rows
    (1, 1, 64, 1.0, "f32"),          # one token: r = 1, every token kept
    (2, 64, 4104, 0.027, "bf16"),    # a width that is not a multiple of 64 (zero-padded rows)
    (1, 30, 40, 0.3, "f32"),
]


@pytest.mark.parametrize("B,Nt,d,scale,dt", TEXT_CASES)
def test_critical_text_parity(B, Nt, d, scale, dt):
    _say(f"[critical-text] B={B} Nt={Nt} d={d} scale={scale} {dt}")
    rng = np.random.default_rng(Nt * 10 + B)
    text = (rng.standard_normal((B, Nt, d)) * scale).astype(np.float32)
    if dt == "bf16":
        text = W.bf16_round(text)
    mask, count, r = run_text(text, dt)
    r_ref, mask_ref, count_ref = oracle.critical_text(text)
    assert rel_err(r, r_ref) <= TOL[dt], rel_err(r, r_ref)
    check_mask(mask, count, r_ref, mask_ref, dt)
    if Nt == 1:
        assert mask.tolist() == [[1]] and count.tolist() == [1]


@pytest.mark.parametrize("wid", [2, 4])
def test_critical_text_workload_falls_back_to_every_row(wid):
    """The workloads' text rows are N(0,1) of width 4096: every softmax row is
    one-hot on its own token, all r equal 1/Nt, and T is every row, on both
    sides."""
    w = W.make_workload(wid, with_kv=False)
    mask, count, r = run_text(w.anchors, w.dtype)
    r_ref, mask_ref, count_ref = oracle.critical_text(w.anchors)
    assert np.all(mask_ref == 1) and np.all(count_ref == w.spec.Nt)
    assert np.all(mask == 1) and np.all(count == w.spec.Nt)
    assert np.all(r == np.float32(1.0 / w.spec.Nt))


def _mask_for(rng, B, Nt, frac):
    m = (rng.random((B, Nt)) < frac).astype(np.int32)
    m[:, rng.integers(0, Nt)] = 1  # at least one row per sample
    return m


@pytest.mark.parametrize("B,Nv,Nt,d,budget,dt", [
    (1, 576, 64, 4096, 192, "bf16"),   # one full-k pass over 16 x 16 tiles
    (16, 300, 40, 1024, 100, "bf16"),  # split-k products
    (1, 200, 9, 256, 50, "f32"),
])
def test_dedup_masked_parity(B, Nv, Nt, d, budget, dt):
    """Only the masked rows are anchors: the oracle is pruning before the LLM
    over those rows alone."""
    from paper_2608_25332_amd import provip
    _say(f"[dedup-masked] B={B} Nv={Nv} Nt={Nt} d={d} budget={budget} {dt}")
    rng = np.random.default_rng(Nv + Nt)
    vis = rng.standard_normal((B, Nv, d)).astype(np.float32)
    anc = rng.standard_normal((B, Nt, d)).astype(np.float32)
    if dt == "bf16":
        vis, anc = W.bf16_round(vis), W.bf16_round(anc)
    m = _mask_for(rng, B, Nt, 0.4)
    g = provip.pv_prune_dedup(to_dev(vis, dt), to_dev(anc, dt), budget, want_merged=False,
                              anchor_mask=torch.from_numpy(m).to("cuda:0"))
    torch.cuda.synchronize()
    score, kept = to_host(g["score"]), to_host(g["kept"])
    for b in range(B):
        rows = anc[b][m[b] == 1]
        p = oracle.maxpool(oracle.center(oracle.cosine(rows, vis[b])))
        assert rel_err(score[b], p) <= TOL[dt], rel_err(score[b], p)
        check_kept(kept[b], p, budget, dt)


def test_dedup_empty_mask_means_every_row():
    from paper_2608_25332_amd import provip
    rng = np.random.default_rng(3)
    vis = W.bf16_round(rng.standard_normal((2, 100, 256)).astype(np.float32))
    anc = W.bf16_round(rng.standard_normal((2, 12, 256)).astype(np.float32))
    vd, ad = to_dev(vis, "bf16"), to_dev(anc, "bf16")
    full = provip.pv_prune_dedup(vd, ad, 30, want_merged=False)
    empty = provip.pv_prune_dedup(vd, ad, 30, want_merged=False,
                                  anchor_mask=torch.zeros((2, 12), dtype=torch.int32,
                                                          device="cuda:0"))
    ones = provip.pv_prune_dedup(vd, ad, 30, want_merged=False,
                                 anchor_mask=torch.ones((2, 12), dtype=torch.int32,
                                                        device="cuda:0"))
    torch.cuda.synchronize()
    for o in (empty, ones):
        assert torch.equal(o["kept"], full["kept"]) and torch.equal(o["score"], full["score"])


@pytest.mark.parametrize("B,H,Nt,N,hd,n_vis,dt", [
    (2, 32, 64, 192, 128, 6, "bf16"),
    (3, 8, 33, 100, 64, 3, "f32"),
])
def test_visual_heads_masked_parity(B, H, Nt, N, hd, n_vis, dt):
    from paper_2608_25332_amd import provip
    _say(f"[visual-heads-masked] B={B} H={H} Nt={Nt} N={N} hd={hd} {dt}")
    rng = np.random.default_rng(H + N)
    q = (rng.standard_normal((B, H, Nt, hd)) * 1.5).astype(np.float32)
    k = (rng.standard_normal((B, H, N, hd)) * 1.5).astype(np.float32)
    if dt == "bf16":
        q, k = W.bf16_round(q), W.bf16_round(k)
    m = _mask_for(rng, B, Nt, 0.5)
    r = provip.pv_visual_heads(to_dev(q, dt), to_dev(k, dt), n_vis,
                               row_mask=torch.from_numpy(m).to("cuda:0"))
    torch.cuda.synchronize()
    heads, conf = to_host(r["heads"]), to_host(r["conf"])
    for b in range(B):
        qb = q[b:b + 1][:, :, m[b] == 1]
        ref_heads, ref_conf = oracle.visual_heads(qb, k[b:b + 1], n_vis)
        assert rel_err(conf[b], ref_conf[0]) <= TOL[dt]
        check_kept(heads[b], ref_conf[0], n_vis, dt)


def test_critical_text_then_dedup():
    """Sec. 4.2 feeding Sec. 4.3 without leaving the GPU: the mask from
    pv_critical_text restricts the anchors of pruning before the LLM."""
    from paper_2608_25332_amd import provip
    rng = np.random.default_rng(11)
    B, Nv, Nt, d, budget = 2, 576, 64, 4096, 192
    vis = W.bf16_round(rng.standard_normal((B, Nv, d)).astype(np.float32))
    text = W.bf16_round((rng.standard_normal((B, Nt, d)) * 0.027).astype(np.float32))
    td = to_dev(text, "bf16")
    ct = provip.pv_critical_text(td)
    g = provip.pv_prune_dedup(to_dev(vis, "bf16"), td, budget, want_merged=False,
                              anchor_mask=ct["mask"])
    torch.cuda.synchronize()
    mask = to_host(ct["mask"])
    assert 0 < mask.sum() < B * Nt
    for b in range(B):
        rows = text[b][mask[b] == 1]
        p = oracle.maxpool(oracle.center(oracle.cosine(rows, vis[b])))
        assert rel_err(to_host(g["score"])[b], p) <= TOL["bf16"]
        check_kept(to_host(g["kept"])[b], p, budget, "bf16")
