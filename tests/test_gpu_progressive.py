"""The progressive schedule in one call (pv_prune_progressive, Sec. 4
Overview): critical text -> pruning before the LLM on the critical rows ->
visual heads and head-aware pruning at a shallow layer -> all-head pruning at
a middle layer, with the compactions between.  Synthetic per-layer queries
and keys stand in for the two pruning layers (no model weights).

Every stage is checked against the oracle given the GPU's previous stage
(each of which is checked in turn); at the tiny fp32 workload the whole chain
must equal the oracle's own chain; and the call must give the bits of the
library's public calls made one after another."""

from __future__ import annotations

import functools
import sys

import numpy as np
import pytest

import oracle
from paper_2608_25332_amd import workloads as W
from parity_util import (TAU, TOL, check_assign_all, check_kept, check_merged, oracle_p,
                         rel_err, to_dev, to_host)

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


@functools.lru_cache(maxsize=None)
def case(wid: int):
    w = W.make_workload(wid)
    q_m, k_m = W.make_middle_layer(w)
    return w, q_m, k_m


def _run(text, vis, q_s, k_s, q_m, k_m, dt, budgets):
    from paper_2608_25332_amd import provip
    N1, n_vis, N2, N3 = budgets
    ins = [to_dev(a, dt) for a in (text, vis, q_s, k_s, q_m, k_m)]
    o = provip.pv_prune_progressive(*ins, N1, n_vis, N2, N3)
    torch.cuda.synchronize()
    return ins, {k: to_host(v) for k, v in o.items() if k != "workspace"}


def check_stages(text, vis, q_s, k_s, q_m, k_m, dt, budgets, g):
    """Each stage of one call's outputs g against the oracle, given the
    GPU's outputs of the stage before."""
    N1, n_vis, N2, N3 = budgets
    B, Nt = text.shape[:2]
    H = q_s.shape[1]
    # 1. critical text (Sec. 4.2): r > mean(r) decides; tokens whose oracle
    # r lies within TAU of the mean may go either way
    r_ref, mask_ref, _ = oracle.critical_text(text)
    for b in range(B):
        if not (mask_ref[b].all() and g["text_mask"][b].all()):
            mean = r_ref[b].mean()
            sure = np.abs(r_ref[b] - mean) > TAU[dt] * np.abs(r_ref[b]).max()
            assert np.array_equal(g["text_mask"][b][sure], mask_ref[b][sure]), b
    for b in range(B):
        rows = np.nonzero(g["text_mask"][b])[0]
        if len(rows) == 0:
            rows = np.arange(Nt)
        # 2. pruning before the LLM on the critical rows (Sec. 4.3)
        p_ref = oracle_p(text[b:b + 1][:, rows], vis[b:b + 1])[0]
        kept1 = g["kept1"][b]
        check_kept(kept1, p_ref, N1, dt)
        assert np.array_equal(g["assign"][b][kept1], np.arange(N1))
        check_assign_all(g["assign"][b], vis[b], kept1, dt)
        check_merged(g["merged"][b], vis[b], kept1, g["assign"][b], np.arange(N1), dt)
        # 3. shallow layer: visual heads over the critical rows, then the
        # score over every row with the GPU's heads (Sec. 4.4)
        ks = k_s[b][:, kept1]
        _, conf_ref = oracle.visual_heads(q_s[b:b + 1][:, :, rows], ks[None], n_vis)
        assert rel_err(g["conf"][b], conf_ref[0]) <= TOL[dt]
        check_kept(g["vis_heads"][b], conf_ref[0], n_vis, dt)
        _, v2 = oracle.head_aware(q_s[b:b + 1], ks[None], g["vis_heads"][b:b + 1], N2)
        assert rel_err(g["score2"][b], v2[0]) <= TOL[dt]
        loc2 = np.searchsorted(kept1, g["kept2"][b])
        assert np.array_equal(kept1[np.minimum(loc2, N1 - 1)], g["kept2"][b]), \
            "kept2 must be retained tokens"
        check_kept(loc2, v2[0], N2, dt)
        assert np.array_equal(g["hidden2"][b], g["merged"][b][loc2])
        # 4. middle layer: every head (the all-head aggregation)
        km = k_m[b][:, g["kept2"][b]]
        _, v3 = oracle.head_aware(q_m[b:b + 1], km[None], np.arange(H, dtype=np.int32)[None], N3)
        assert rel_err(g["score3"][b], v3[0]) <= TOL[dt]
        loc3 = np.searchsorted(g["kept2"][b], g["kept3"][b])
        assert np.array_equal(g["kept2"][b][np.minimum(loc3, N2 - 1)], g["kept3"][b])
        check_kept(loc3, v3[0], N3, dt)
        assert np.array_equal(g["hidden3"][b], g["hidden2"][b][loc3])


@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_progressive_against_oracle(wid):
    w, q_m, k_m = case(wid)
    budgets = W.progressive_budgets(w.spec)
    _say(f"[progressive] workload {wid} ({w.spec.name}) budgets {budgets}")
    _, g = _run(w.anchors, w.vis, w.q, w.k_full, q_m, k_m, w.dtype, budgets)
    check_stages(w.anchors, w.vis, w.q, w.k_full, q_m, k_m, w.dtype, budgets, g)


def test_progressive_tiny_whole_chain_is_the_oracles():
    """The tiny fp32 workload has no near ties: every output of the call is
    the oracle's own chain (critical text -> masked dedup -> visual heads ->
    head-aware -> all heads)."""
    w, q_m, k_m = case(1)
    N1, n_vis, N2, N3 = W.progressive_budgets(w.spec)
    _, g = _run(w.anchors, w.vis, w.q, w.k_full, q_m, k_m, "f32", (N1, n_vis, N2, N3))
    _, mask, _ = oracle.critical_text(w.anchors)
    rows = np.nonzero(mask[0])[0]
    ref = oracle.dedup(w.anchors[:, rows], w.vis, N1)
    assert np.array_equal(g["kept1"], ref["kept"]) and np.array_equal(g["assign"], ref["assign"])
    assert np.max(np.abs(g["merged"] - ref["merged"])) <= 1e-5 * np.max(np.abs(ref["merged"]))
    ks = w.k_full[0][:, ref["kept"][0]][None]
    heads, _ = oracle.visual_heads(w.q[:, :, rows], ks, n_vis)
    assert np.array_equal(g["vis_heads"], heads)
    k2, _ = oracle.head_aware(w.q, ks, heads, N2)
    tok2 = ref["kept"][0][k2[0]]
    assert np.array_equal(g["kept2"][0], tok2)
    km = k_m[0][:, tok2][None]
    k3, _ = oracle.head_aware(q_m, km, np.arange(w.spec.H, dtype=np.int32)[None], N3)
    assert np.array_equal(g["kept3"][0], tok2[k3[0]])
    want3 = g["merged"][0][k2[0]][k3[0]]
    assert np.array_equal(g["hidden3"][0], want3)


PROG_EDGE = [
    # (B, Nv, Nt, d, H, hd, N1, n_vis, N2, N3, dtype, peaked text rows)
    (2, 300, 20, 256, 8, 64, 100, 3, 40, 10, "bf16", True),
    (1, 90, 7, 128, 4, 128, 40, 1, 40, 1, "f32", True),       # budget2 = budget1, budget3 = 1
    (3, 200, 33, 512, 6, 128, 64, 6, 20, 20, "bf16", False),   # every head visual, N3 = N2
    (1, 1200, 100, 1024, 16, 128, 400, 6, 130, 65, "bf16", True),
    (2, 250, 24, 520, 8, 72, 80, 4, 30, 12, "bf16", True),   # padded widths
]


@pytest.mark.parametrize("B,Nv,Nt,d,H,hd,N1,nv,N2,N3,dt,peaked", PROG_EDGE)
def test_progressive_edges(B, Nv, Nt, d, H, hd, N1, nv, N2, N3, dt, peaked):
    _say(f"[progressive-edge] B={B} Nv={Nv} Nt={Nt} d={d} H={H} hd={hd} "
         f"budgets {N1}/{nv}/{N2}/{N3} {dt} peaked={peaked}")
    rng = np.random.default_rng(B * 31 + Nv + N1)
    f = (lambda a: W.bf16_round(a)) if dt == "bf16" else (lambda a: a)
    text = rng.standard_normal((B, Nt, d)).astype(np.float32)
    if peaked:
        # text rows of unequal norm: the critical set is a strict subset
        text *= rng.uniform(0.05, 0.2, size=(B, Nt, 1)).astype(np.float32)
    text = f(text)
    vis = f(rng.standard_normal((B, Nv, d)).astype(np.float32))
    q_s = f((rng.standard_normal((B, H, Nt, hd)) * 1.5).astype(np.float32))
    k_s = f((rng.standard_normal((B, H, Nv, hd)) * 1.5).astype(np.float32))
    q_m = f((rng.standard_normal((B, H, Nt, hd)) * 1.5).astype(np.float32))
    k_m = f((rng.standard_normal((B, H, Nv, hd)) * 1.5).astype(np.float32))
    budgets = (N1, nv, N2, N3)
    _, g = _run(text, vis, q_s, k_s, q_m, k_m, dt, budgets)
    if peaked:
        assert 0 < g["text_mask"].sum() < B * Nt
    check_stages(text, vis, q_s, k_s, q_m, k_m, dt, budgets, g)


def test_progressive_equals_the_calls_in_turn():
    """The one call gives the bits of the public calls made one after
    another on the same inputs."""
    from paper_2608_25332_amd import provip
    w, q_m, k_m = case(2)
    N1, n_vis, N2, N3 = W.progressive_budgets(w.spec)
    ins, g = _run(w.anchors, w.vis, w.q, w.k_full, q_m, k_m, "bf16", (N1, n_vis, N2, N3))
    text, vis, q_s, k_s, qm, km_all = ins
    ct = provip.pv_critical_text(text)
    d1 = provip.pv_prune_dedup(vis, text, N1, want_score=False, anchor_mask=ct["mask"])
    ks = provip.pv_prune_gather(k_s, d1["kept"])
    vh = provip.pv_visual_heads(q_s, ks, n_vis, row_mask=ct["mask"])
    h2 = provip.pv_prune_head_aware(q_s, ks, vh["heads"], N2)
    loc2 = h2["kept"]
    kept2 = torch.gather(d1["kept"], 1, loc2.long()).to(torch.int32)
    hid2 = provip.pv_prune_gather(d1["merged"], loc2)
    km = provip.pv_prune_gather(km_all, kept2)
    all_heads = np.tile(np.arange(w.spec.H, dtype=np.int32), (w.spec.B, 1))
    h3 = provip.pv_prune_head_aware(qm, km, all_heads, N3)
    kept3 = torch.gather(kept2, 1, h3["kept"].long()).to(torch.int32)
    hid3 = provip.pv_prune_gather(hid2, h3["kept"])
    torch.cuda.synchronize()
    pairs = {"text_mask": ct["mask"], "kept1": d1["kept"], "assign": d1["assign"],
             "merged": d1["merged"], "vis_heads": vh["heads"], "conf": vh["conf"],
             "kept2": kept2, "score2": h2["score"], "hidden2": hid2, "kept3": kept3,
             "score3": h3["score"], "hidden3": hid3}
    for name, t in pairs.items():
        assert np.array_equal(g[name], to_host(t)), name
