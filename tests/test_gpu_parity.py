"""HIP path vs the CPU oracle, element by element, on the seeded workloads.

All calls go through the C ABI (ctypes binding).  Every workload is checked
in full: p and the kept set of every sample, the nearest kept token of every
pruned row (the oracle given the GPU's kept list) and every merged slot (the
oracle given the GPU's assignment).  At the large workloads the oracle runs
over row ranges in parallel threads (the same arithmetic as one call).
"""

from __future__ import annotations

import functools
import sys

import numpy as np
import pytest

import oracle
from paper_2608_25332_amd import workloads as W
from parity_util import (TOL, check_assign_rows, check_dedup_sample, check_kept, check_merged,
                         oracle_p_workload, rel_err, to_dev, to_host)

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
def workload(wid: int, with_kv: bool = True):
    return W.make_workload(wid, with_kv=with_kv)


def run_dedup(vis_np, anc_np, dtype, budget):
    from paper_2608_25332_amd import provip
    vis = to_dev(vis_np, dtype)
    anc = to_dev(anc_np, dtype)
    r = provip.pv_prune_dedup(vis, anc, budget)
    torch.cuda.synchronize()
    return {k: (to_host(v) if hasattr(v, "cpu") else v) for k, v in r.items() if k != "workspace"}


# --------------------------------------------------------------- dedup ------

@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_dedup_parity(wid):
    w = workload(wid, with_kv=False)
    dt = w.dtype
    _say(f"[dedup] workload {wid} {w.spec.name} B={w.spec.B} Nv={w.spec.Nv} d={w.spec.d}")
    g = run_dedup(w.vis, w.anchors, dt, w.N1)
    B = w.spec.B
    for b in range(B):
        kept = g["kept"][b]
        assert np.all(np.diff(kept) > 0) and kept.shape == (w.N1,)
        # kept tokens are their own centroids; every token has a valid slot
        assert np.array_equal(g["assign"][b][kept], np.arange(w.N1))
        assert g["assign"][b].min() >= 0 and g["assign"][b].max() < w.N1
    p_ref = oracle_p_workload(wid, w.anchors, w.vis)
    ex_k = ex_a = 0
    for b in range(B):
        k, a = check_dedup_sample(g, b, w.vis[b], p_ref[b], w.N1, dt)
        ex_k += k
        ex_a += a
    _say(f"[dedup] workload {wid}: ok on all {B} samples, every pruned row and slot; "
         f"{ex_k} near-tie tokens, {ex_a} near-tie rows exempt")


def test_dedup_tiny_exact_against_full_oracle():
    w = workload(1, with_kv=False)
    g = run_dedup(w.vis, w.anchors, "f32", w.N1)
    ref = oracle.dedup(w.anchors, w.vis, w.N1)
    assert np.array_equal(g["kept"], ref["kept"])
    assert np.array_equal(g["assign"], ref["assign"])
    assert rel_err(g["merged"], ref["merged"]) <= 1e-5


def test_dedup_twins_on_gpu():
    """Planted exact duplicates: bit-identical p; if the higher twin is kept
    the lower one is too; a pruned twin of a kept token is absorbed by it."""
    w = workload(1, with_kv=False)
    for dt in ("f32", "bf16"):
        vis = w.vis if dt == "f32" else W.bf16_round(w.vis)
        anc = w.anchors if dt == "f32" else W.bf16_round(w.anchors)
        g = run_dedup(vis, anc, dt, w.N1)
        kept = set(g["kept"][0].tolist())
        for a, b in w.dup_pairs:
            assert g["score"][0, a] == g["score"][0, b], (dt, a, b)
            if b in kept:
                assert a in kept
            if a in kept and b not in kept:
                assert g["assign"][0, b] == list(g["kept"][0]).index(a)


def test_dedup_deterministic():
    w = workload(2, with_kv=False)
    a = run_dedup(w.vis, w.anchors, "bf16", w.N1)
    b = run_dedup(w.vis, w.anchors, "bf16", w.N1)
    for k in ("kept", "score", "assign", "merged"):
        assert np.array_equal(a[k], b[k]), k


def test_timed_reps_leave_results_unchanged():
    """The profiling variants with every kernel launched several times give
    the results of one launch (no kernel reads what it writes)."""
    from paper_2608_25332_amd import provip
    w = workload(2)
    vis, anc = to_dev(w.vis, "bf16"), to_dev(w.anchors, "bf16")
    a = provip.pv_prune_dedup(vis, anc, w.N1)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(8)]
    for e in ev:  # torch creates the HIP event on its first record
        e.record()
    b = provip.pv_prune_dedup(vis, anc, w.N1, events=ev, reps=3)
    torch.cuda.synchronize()
    assert b["n_kernels"] == len(b["kernel_names"]) >= 5
    for k in ("kept", "score", "assign", "merged"):
        assert torch.equal(a[k], b[k]), k
    q, kf = to_dev(w.q, "bf16"), to_dev(w.k_full, "bf16")
    k1 = provip.pv_prune_gather(kf, a["kept"])
    h1 = provip.pv_prune_head_aware(q, k1, w.heads, w.N2)
    ev2 = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in ev2:
        e.record()
    h2 = provip.pv_prune_head_aware(q, k1, w.heads, w.N2, events=ev2, reps=4)
    torch.cuda.synchronize()
    assert h2["kernel_names"] == ["score_partial", "score_select"]
    for k in ("kept", "score"):
        assert torch.equal(h1[k], h2[k]), k


@pytest.mark.parametrize("wid", [1, 2, 4, 5])
def test_dedup_split_matches_single_stream(wid):
    """pv_prune_dedup_split (merge branch on a second stream) gives the bits
    of pv_prune_dedup once merged_done has completed."""
    from paper_2608_25332_amd import provip
    w = workload(wid, with_kv=False)
    dt = w.dtype
    vis, anc = to_dev(w.vis, dt), to_dev(w.anchors, dt)
    a = provip.pv_prune_dedup(vis, anc, w.N1)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    sel, done = torch.cuda.Event(), torch.cuda.Event()
    sel.record()
    done.record()
    b = provip.pv_prune_dedup(vis, anc, w.N1, split=(side, sel, done))
    torch.cuda.current_stream().wait_event(done)
    torch.cuda.synchronize()
    for k in ("kept", "score", "assign", "merged"):
        assert torch.equal(a[k], b[k]), k


# full-k Gram shapes for the split call, whose Gram takes the 256-row tiles
# with loads two chunks ahead: one chunk (d = 64 bf16), one kept tile, two
# kept tiles in fp32, padded rows, ragged tiles in both directions
SPLIT_EDGE = [
    (128, 300, 4, 64, 100, "bf16"),
    (64, 600, 4, 128, 200, "f32"),
    (64, 600, 4, 1000, 200, "bf16"),
    (8, 1700, 16, 256, 500, "bf16"),
    (16, 900, 8, 384, 300, "bf16"),
]


@pytest.mark.parametrize("B,Nv,Nt,d,budget,dt", SPLIT_EDGE)
def test_dedup_split_edges(B, Nv, Nt, d, budget, dt):
    """The split call's Gram against the single-stream call (same bits) and
    its assignment against the oracle on every pruned row of the first and
    last sample."""
    from paper_2608_25332_amd import provip
    _say(f"[dedup-split-edge] B={B} Nv={Nv} Nt={Nt} d={d} budget={budget} {dt}")
    rng = np.random.default_rng(Nv * 11 + d)
    vis = rng.standard_normal((B, Nv, d)).astype(np.float32)
    anc = rng.standard_normal((B, Nt, d)).astype(np.float32)
    if dt == "bf16":
        vis, anc = W.bf16_round(vis), W.bf16_round(anc)
    dv, da = to_dev(vis, dt), to_dev(anc, dt)
    a = provip.pv_prune_dedup(dv, da, budget)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    sel, done = torch.cuda.Event(), torch.cuda.Event()
    sel.record()
    done.record()
    b = provip.pv_prune_dedup(dv, da, budget, split=(side, sel, done))
    torch.cuda.current_stream().wait_event(done)
    torch.cuda.synchronize()
    for k in ("kept", "score", "assign", "merged"):
        assert torch.equal(a[k], b[k]), k
    kept_all, assign_all = to_host(b["kept"]), to_host(b["assign"])
    for bb in sorted({0, B - 1}):
        kept = kept_all[bb]
        pruned = np.setdiff1d(np.arange(Nv), kept)
        check_assign_rows(assign_all[bb], vis[bb], kept, pruned, dt)


DEDUP_EDGE = [
    # (B, Nv, Nt, d, budget, dtype)
    (1, 17, 1, 64, 5, "f32"),
    (2, 33, 3, 128, 33, "bf16"),     # budget == Nv: identity, nothing pruned
    (3, 70, 20, 192, 1, "bf16"),     # budget == 1
    (1, 300, 37, 256, 129, "bf16"),  # ragged everywhere
    (2, 1000, 130, 320, 333, "bf16"),
    (1, 5, 2, 64, 4, "f32"),
    # k ranges that are not a multiple of the unroll depth (wave slices with
    # 0 or 1 windows): regression cases for masked-off MFMA blocks
    (1, 40, 4, 128, 1, "bf16"),
    (1, 40, 4, 192, 1, "bf16"),
    (1, 40, 4, 256, 3, "bf16"),
    (2, 40, 4, 320, 7, "f32"),
    # split-k cosine (batches too large for the full-k small-input pass),
    # ragged tiles in both directions
    (64, 200, 33, 1024, 70, "bf16"),
    (48, 150, 5, 2048, 40, "f32"),
    (8, 1000, 130, 256, 300, "bf16"),
    (2, 1500, 100, 2048, 400, "bf16"),
    (1, 1200, 70, 2048, 300, "f32"),
    # wide split-k Gram tiles (128 x 96), ragged in both directions (three
    # cases above take them too: 64 x 200, 2 x 1500 and the fp32 1 x 1200)
    (12, 500, 64, 4096, 150, "bf16"),
    # member-list merge: 10-37 members in every slot (the many-member path,
    # four rows per wave in flight, ragged last rounds), then 2-16 members
    # (both paths in one launch)
    (2, 400, 8, 256, 20, "f32"),
    (3, 401, 8, 192, 50, "bf16"),
    # full-k Gram tiles: one kept tile (slot written directly), and two kept
    # tiles in fp32 (per-tile candidates merged by gram_finish); one, two and
    # three 128-byte chunks per row (the load ring's short starts)
    (128, 300, 4, 64, 100, "bf16"),
    (64, 600, 4, 128, 200, "f32"),
    (128, 300, 4, 128, 100, "bf16"),
    (128, 300, 4, 192, 100, "bf16"),
    # full-k Gram edge tiles where whole matrix waves lie past the last pruned
    # row (136 of 256) and the last kept slot (64 of 128): they skip their
    # MFMAs
    (128, 200, 4, 128, 64, "bf16"),
    (128, 200, 4, 64, 64, "f32"),
    # split-k cosine on 128 x 128 tiles at the boundary (65 anchors, 512 tokens)
    (16, 512, 65, 2048, 100, "bf16"),
    # four-token slice reduction at its smallest (8 tokens, many anchors)
    (64, 8, 130, 4096, 3, "f32"),
    # merge through bucketed member lists (narrow rows, many slots)
    (1, 1000, 8, 64, 70, "bf16"),
    (2, 700, 5, 128, 200, "f32"),
    # widths that are multiples of 8 but not of the streamed chunk: the rows
    # are copied zero-padded into the workspace first
    (2, 300, 20, 4104, 100, "bf16"),
    (1, 200, 9, 4104, 50, "f32"),
    (1, 50, 3, 8, 10, "f32"),
    (3, 90, 12, 72, 30, "bf16"),
    (16, 200, 64, 520, 64, "bf16"),       # split-k cosine on padded rows
    (64, 600, 4, 1000, 200, "bf16"),      # full-k Gram tiles on padded rows
]


@pytest.mark.parametrize("B,Nv,Nt,d,budget,dt", DEDUP_EDGE)
def test_dedup_edges(B, Nv, Nt, d, budget, dt):
    _say(f"[dedup-edge] B={B} Nv={Nv} Nt={Nt} d={d} budget={budget} {dt}")
    rng = np.random.default_rng(Nv * 7 + Nt)
    vis = rng.standard_normal((B, Nv, d)).astype(np.float32)
    anc = rng.standard_normal((B, Nt, d)).astype(np.float32)
    if dt == "bf16":
        vis, anc = W.bf16_round(vis), W.bf16_round(anc)
    g = run_dedup(vis, anc, dt, budget)
    g2 = run_dedup(vis, anc, dt, budget)
    for key in ("kept", "score", "assign", "merged"):
        assert np.array_equal(g[key], g2[key]), f"two calls differ in {key}"
    for b in range(B):
        p = oracle.maxpool(oracle.center(oracle.cosine(anc[b], vis[b])))
        assert rel_err(g["score"][b], p) <= TOL[dt]
        check_kept(g["kept"][b], p, budget, dt)
        kept = g["kept"][b]
        pruned = np.setdiff1d(np.arange(Nv), kept)
        if len(pruned):
            check_assign_rows(g["assign"][b], vis[b], kept, pruned, dt)
        check_merged(g["merged"][b], vis[b], kept, g["assign"][b], np.arange(budget), dt)
        if budget == Nv:
            assert np.array_equal(kept, np.arange(Nv))
            assert np.array_equal(g["merged"][b], vis[b])


def test_dedup_one_slot_takes_almost_everything():
    """Identical visual tokens: every pruned token ties on cosine 1 and goes
    to slot 0 (lowest slot), whose member list then exceeds one 4096-entry
    round of the merge."""
    rng = np.random.default_rng(9)
    row = W.bf16_round(rng.standard_normal(64).astype(np.float32))
    vis = np.ascontiguousarray(np.broadcast_to(row, (1, 5000, 64)), np.float32)
    anc = W.bf16_round(rng.standard_normal((1, 3, 64)).astype(np.float32))
    g = run_dedup(vis, anc, "bf16", 40)
    assert np.array_equal(g["kept"][0], np.arange(40))
    want = np.zeros(5000, np.int32)
    want[:40] = np.arange(40)
    assert np.array_equal(g["assign"][0], want)
    check_merged(g["merged"][0], vis[0], g["kept"][0], g["assign"][0], np.arange(40), "bf16")


@pytest.mark.parametrize("B,Nv,Nt,d,dt", [
    (1, 40, 4, 64, "f32"),         # one full-k pass over 16 x 16 tiles
    (130, 70, 100, 128, "bf16"),   # split-k products, many samples
    (1, 1500, 100, 2048, "bf16"),  # split-k products, long rows
])
def test_dedup_zero_vectors(B, Nv, Nt, d, dt):
    """A zero visual token or anchor has cosine 0 to everything (each way
    the cosines are formed)."""
    _say(f"[dedup-zero] B={B} Nv={Nv} Nt={Nt} d={d} {dt}")
    rng = np.random.default_rng(5)
    vis = rng.standard_normal((B, Nv, d)).astype(np.float32)
    anc = rng.standard_normal((B, Nt, d)).astype(np.float32)
    if dt == "bf16":
        vis, anc = W.bf16_round(vis), W.bf16_round(anc)
    vis[:, 7] = 0.0
    anc[:, 2] = 0.0
    g = run_dedup(vis, anc, dt, 10)
    for b in range(min(B, 3)):
        p = oracle.maxpool(oracle.center(oracle.cosine(anc[b], vis[b])))
        assert rel_err(g["score"][b], p) <= TOL[dt]
        check_kept(g["kept"][b], p, 10, dt)


# ----------------------------------------------------------- head-aware -----

def _subset_keys(w, n, seed):
    rng = np.random.default_rng(seed)
    idx = np.stack([np.sort(rng.choice(w.spec.Nv, n, replace=False)) for _ in range(w.spec.B)])
    k = np.stack([w.k_full[b][:, idx[b]] for b in range(w.spec.B)])
    return np.ascontiguousarray(k)


def run_head(q_np, k_np, heads, dtype, budget):
    from paper_2608_25332_amd import provip
    q = to_dev(q_np, dtype)
    k = to_dev(k_np, dtype)
    r = provip.pv_prune_head_aware(q, k, heads, budget)
    torch.cuda.synchronize()
    return to_host(r["kept"]), to_host(r["score"])


@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_head_aware_parity(wid):
    w = workload(wid)
    dt = w.dtype
    _say(f"[head-aware] workload {wid} heads={w.heads.tolist()[:2]}")
    k1 = _subset_keys(w, w.N1, 200 + wid)
    kept, v = run_head(w.q, k1, w.heads, dt, w.N2)
    ref_kept, ref_v = oracle.head_aware(w.q, k1, w.heads, w.N2)
    assert rel_err(v, ref_v) <= TOL[dt], rel_err(v, ref_v)
    for b in range(w.spec.B):
        check_kept(kept[b], ref_v[b], w.N2, dt)
        assert abs(float(np.sum(v[b], dtype=np.float64)) - 1.0) < 1e-4


@pytest.mark.parametrize("wid", [2, 4])
def test_head_aware_all_heads(wid):
    """Every head selected: the all-head aggregation of the middle layer."""
    w = workload(wid)
    k1 = _subset_keys(w, w.N1, 300 + wid)
    heads = np.tile(np.arange(w.spec.H, dtype=np.int32), (w.spec.B, 1))
    kept, v = run_head(w.q, k1, heads, w.dtype, w.N2)
    ref_kept, ref_v = oracle.head_aware(w.q, k1, heads, w.N2)
    assert rel_err(v, ref_v) <= TOL[w.dtype]
    for b in range(w.spec.B):
        check_kept(kept[b], ref_v[b], w.N2, w.dtype)


HEAD_EDGE = [
    # (B, H, Nt, N, hd, heads per sample, budget, dtype)
    (1, 2, 1, 1, 32, 1, 1, "f32"),
    (1, 3, 1, 15, 64, 2, 15, "bf16"),
    (2, 4, 17, 17, 64, 3, 5, "bf16"),
    (3, 8, 33, 100, 128, 8, 40, "bf16"),
    (1, 4, 16, 64, 256, 2, 16, "bf16"),
    (2, 4, 5, 50, 96, 1, 7, "f32"),
    (1, 2, 200, 2100, 128, 2, 600, "bf16"),   # keys streamed twice
    (2, 3, 40, 1500, 128, 2, 200, "bf16"),    # 24 chunks of logits held in registers
    (1, 4, 50, 900, 64, 2, 100, "bf16"),      # 15 chunks, ragged, logits held
    (2, 2, 20, 700, 32, 1, 50, "f32"),        # 11 chunks, fp32, logits held
    (1, 2, 20, 600, 256, 1, 100, "bf16"),     # wide head, streamed twice
    (1, 2, 16, 130, 256, 2, 30, "f32"),       # widest head, logits kept
    (1, 2, 16, 300, 256, 1, 30, "f32"),       # widest head, streamed twice
    (2, 3, 40, 70, 160, 2, 9, "bf16"),
    (1, 2, 33, 257, 224, 2, 64, "f32"),
    (40, 16, 80, 64, 64, 16, 20, "bf16"),     # 640 head-list entries of 16-row blocks: two launches
    (1, 2, 16, 9000, 256, 1, 500, "f32"),     # column sums flushed from registers
    (1, 1, 9, 12100, 224, 1, 900, "f32"),     # the same, 14 pieces per key row
    # one workgroup per (head, sample) once there are >= 128 of them
    (32, 8, 64, 256, 128, 4, 60, "bf16"),     # four full key chunks
    (64, 4, 33, 70, 64, 2, 10, "f32"),        # ragged rows (an idle wave) and keys
    (128, 2, 1, 1, 32, 1, 1, "f32"),          # one row, one key
    (130, 3, 50, 200, 64, 1, 20, "bf16"),
    (16, 32, 64, 192, 128, 32, 64, "bf16"),   # every head of the LLaVA-1.5 layer
    # split over 64-key chunks (long key lists on few head-sample pairs)
    (1, 4, 128, 960, 128, 4, 320, "bf16"),    # one hi-res sample
    (2, 5, 128, 1152, 128, 5, 512, "bf16"),   # the 13B batch
    (3, 4, 17, 300, 64, 2, 50, "f32"),        # last chunk of 44 keys, 256-byte fp32 rows
    (1, 3, 1, 257, 64, 1, 10, "bf16"),        # one row; last chunk of one key
    (2, 8, 200, 700, 128, 3, 99, "bf16"),     # four passes of 64 rows, ragged
    # the 16-row blocks at long key lists (enough blocks to fill the chip)
    (16, 4, 64, 1500, 128, 4, 200, "bf16"),   # 24 chunks of logits held in registers
    (10, 2, 200, 2100, 128, 2, 600, "bf16"),  # keys streamed twice
    # head widths that are multiples of 8 but not of 32 (zero-padded copies;
    # the scale stays 1 / sqrt(hd))
    (2, 4, 17, 100, 72, 2, 30, "bf16"),
    (1, 3, 20, 300, 80, 2, 50, "f32"),
    (2, 8, 64, 960, 112, 4, 200, "bf16"),     # split form on padded rows
    (1, 2, 5, 33, 8, 1, 5, "f32"),
    (40, 8, 64, 192, 80, 4, 64, "bf16"),      # whole-head form on padded rows
    (3, 4, 30, 70, 40, "all", 20, "bf16"),    # every head
]


def score_form(B, H, Nt, N, hd, nh, dt):
    """The score form the library picks (its rule, restated for the test
    log): whole-head, split over key chunks, or 16-row blocks."""
    nks = hd * (2 if dt == "bf16" else 4) // 64
    if nks in (2, 4) and H <= 256 and Nt <= 64 and N <= 256 and B * nh >= 128:
        return "whole-head"
    if nks in (2, 4) and N > 256 and ((Nt + 15) // 16) * nh * B < 256:
        return "split"
    return "row-blocks"


@pytest.mark.parametrize("B,H,Nt,N,hd,nh,budget,dt", HEAD_EDGE)
def test_head_aware_edges(B, H, Nt, N, hd, nh, budget, dt):
    form = score_form(B, H, Nt, N, (hd + 31) // 32 * 32, H if nh == "all" else nh, dt)
    _say(f"[head-edge] B={B} H={H} Nt={Nt} N={N} hd={hd} nh={nh} budget={budget} {dt} ({form})")
    rng = np.random.default_rng(B * 1000 + N)
    q = (rng.standard_normal((B, H, Nt, hd)) * 1.5).astype(np.float32)
    k = (rng.standard_normal((B, H, N, hd)) * 1.5).astype(np.float32)
    if dt == "bf16":
        q, k = W.bf16_round(q), W.bf16_round(k)
    if nh == "all":
        heads = np.tile(np.arange(H, dtype=np.int32), (B, 1))
    else:
        heads = np.stack([rng.permutation(H)[:nh] for _ in range(B)]).astype(np.int32)
    kept, v = run_head(q, k, heads, dt, budget)
    _, ref_v = oracle.head_aware(q, k, heads, budget)
    assert rel_err(v, ref_v) <= TOL[dt]
    for b in range(B):
        check_kept(kept[b], ref_v[b], budget, dt)


LARGE_BATCH_CASES = [
    # (B, H, Nt, N, hd, heads per sample, budget, dtype): batches of 520 to
    # 2400 (head, sample) pairs
    (160, 8, 64, 192, 128, 4, 64, "bf16"),
    (300, 4, 40, 130, 64, 2, 20, "bf16"),    # ragged rows and keys, 2 workgroups per CU
    (130, 8, 20, 100, 64, 4, 30, "f32"),
    (600, 4, 64, 192, 128, 4, 64, "bf16"),   # 2400 pairs: two launches of host lists
    (512, 2, 1, 1, 128, 1, 1, "bf16"),       # one row, one key
]


@pytest.mark.parametrize("B,H,Nt,N,hd,nh,budget,dt", LARGE_BATCH_CASES)
def test_head_aware_large_batches(B, H, Nt, N, hd, nh, budget, dt):
    """Large batches: host head lists (several launches of bounded lists)
    give the bits of device head lists (one launch), and both match the
    oracle."""
    from paper_2608_25332_amd import provip
    _say(f"[head-large] B={B} H={H} Nt={Nt} N={N} hd={hd} nh={nh} budget={budget} {dt}")
    rng = np.random.default_rng(B * 31 + N)
    q = (rng.standard_normal((B, H, Nt, hd)) * 1.5).astype(np.float32)
    k = (rng.standard_normal((B, H, N, hd)) * 1.5).astype(np.float32)
    if dt == "bf16":
        q, k = W.bf16_round(q), W.bf16_round(k)
    heads = np.stack([rng.permutation(H)[:nh] for _ in range(B)]).astype(np.int32)
    qd, kd = to_dev(q, dt), to_dev(k, dt)
    a = provip.pv_prune_head_aware(qd, kd, heads, budget)
    b = provip.pv_prune_head_aware(qd, kd, torch.from_numpy(heads).to("cuda:0"), budget)
    torch.cuda.synchronize()
    assert torch.equal(a["score"], b["score"]) and torch.equal(a["kept"], b["kept"])
    sel = np.arange(0, B, max(1, B // 40))  # the oracle on a spread of samples
    _, ref_v = oracle.head_aware(q[sel], k[sel], heads[sel], budget)
    v, kept = to_host(a["score"])[sel], to_host(a["kept"])[sel]
    assert rel_err(v, ref_v) <= TOL[dt], rel_err(v, ref_v)
    for i in range(len(sel)):
        check_kept(kept[i], ref_v[i], budget, dt)


def test_head_aware_large_batch_in_model():
    """The in-model domain on a batch of 544 (head, sample) pairs, against the
    oracle."""
    from paper_2608_25332_amd import provip
    rng = np.random.default_rng(21)
    B, H, Nt, N, hd, nh = 136, 8, 64, 192, 128, 4
    q = W.bf16_round((rng.standard_normal((B, H, Nt, hd)) * 1.5).astype(np.float32))
    k = W.bf16_round((rng.standard_normal((B, H, N, hd)) * 1.5).astype(np.float32))
    heads = np.stack([rng.permutation(H)[:nh] for _ in range(B)]).astype(np.int32)
    # log-sum-exp of each row's scaled logits over 50 synthetic non-visual keys
    ko = rng.standard_normal((B, H, 50, hd)) * 1.5
    lg = np.einsum("bhid,bhjd->bhij", q.astype(np.float64), ko) / np.sqrt(hd)
    mx = lg.max(-1, keepdims=True)
    lse = (mx[..., 0] + np.log(np.exp(lg - mx).sum(-1))).astype(np.float32)
    r = provip.pv_prune_head_aware(to_dev(q, "bf16"), to_dev(k, "bf16"), heads, 30,
                                   row_lse=torch.from_numpy(lse).to("cuda:0"))
    torch.cuda.synchronize()
    v, kept = to_host(r["score"]), to_host(r["kept"])
    ref_kept, ref_v = oracle.head_aware_in_model(q, k, heads, lse.astype(np.float64), 30)
    assert rel_err(v, ref_v) <= TOL["bf16"], rel_err(v, ref_v)
    for b in range(B):
        check_kept(kept[b], ref_v[b], 30, "bf16")


def test_head_aware_duplicate_keys_tie():
    """Exact duplicate keys get bit-identical v, and the lower index wins."""
    rng = np.random.default_rng(9)
    q = rng.standard_normal((1, 2, 8, 64)).astype(np.float32)
    k = rng.standard_normal((1, 2, 40, 64)).astype(np.float32)
    k[:, :, 30] = k[:, :, 4]
    k[:, :, 4] *= 3.0   # make token 4 (and its twin 30) important
    k[:, :, 30] = k[:, :, 4]
    kept, v = run_head(q, k, [[0, 1]], "f32", 1)
    assert v[0, 4] == v[0, 30]
    if v[0].argmax() in (4, 30):
        assert kept[0].tolist() == [4]


# --------------------------------------------------------------- gather -----

def test_gather_bit_exact():
    from paper_2608_25332_amd import provip
    rng = np.random.default_rng(3)
    B, H, N, hd, D, k = 2, 8, 300, 128, 4096, 97
    hid = torch.from_numpy(rng.standard_normal((B, N, D)).astype(np.float32)).to("cuda:0").bfloat16()
    kv = torch.from_numpy(rng.standard_normal((B, H, N, hd)).astype(np.float32)).to("cuda:0").bfloat16()
    idx_np = np.stack([np.sort(rng.choice(N, k, replace=False)) for _ in range(B)]).astype(np.int32)
    idx = torch.from_numpy(idx_np).to("cuda:0")
    oh = provip.pv_prune_gather(hid, idx)
    ok = provip.pv_prune_gather(kv, idx)
    torch.cuda.synchronize()
    hb = hid.view(torch.int16).cpu().numpy()
    kb = kv.view(torch.int16).cpu().numpy()
    assert np.array_equal(oh.view(torch.int16).cpu().numpy(), oracle.gather(hb, idx_np))
    assert np.array_equal(ok.view(torch.int16).cpu().numpy(), oracle.gather(kb, idx_np))


def test_gather_batch_bit_exact():
    """Hidden, K and V (different row sizes) in one launch."""
    from paper_2608_25332_amd import provip
    rng = np.random.default_rng(4)
    B, H, N, hd, D, k = 3, 4, 77, 64, 512, 31
    hid = torch.from_numpy(rng.standard_normal((B, N, D)).astype(np.float32)).to("cuda:0")
    kk = torch.from_numpy(rng.standard_normal((B, H, N, hd)).astype(np.float32)).to("cuda:0").bfloat16()
    vv = torch.from_numpy(rng.standard_normal((B, H, N, hd)).astype(np.float32)).to("cuda:0").bfloat16()
    idx_np = np.stack([np.sort(rng.choice(N, k, replace=False)) for _ in range(B)]).astype(np.int32)
    idx = torch.from_numpy(idx_np).to("cuda:0")
    oh, ok, ov = provip.pv_prune_gather_batch([hid, kk, vv], idx)
    torch.cuda.synchronize()
    assert np.array_equal(oh.cpu().numpy(), oracle.gather(hid.cpu().numpy(), idx_np))
    assert np.array_equal(ok.view(torch.int16).cpu().numpy(), oracle.gather(kk.view(torch.int16).cpu().numpy(), idx_np))
    assert np.array_equal(ov.view(torch.int16).cpu().numpy(), oracle.gather(vv.view(torch.int16).cpu().numpy(), idx_np))


def test_gather_out_of_range_rows_are_zero():
    from paper_2608_25332_amd import provip
    src = torch.arange(4 * 8, dtype=torch.float32, device="cuda:0").reshape(1, 8, 4) + 1
    idx = torch.tensor([[0, 9, -1, 7]], dtype=torch.int32, device="cuda:0")
    out = provip.pv_prune_gather(src, idx).cpu().numpy()
    s = src.cpu().numpy()
    assert np.array_equal(out[0, 0], s[0, 0]) and np.array_equal(out[0, 3], s[0, 7])
    assert np.all(out[0, 1] == 0) and np.all(out[0, 2] == 0)


# ------------------------------------------------------------- pipeline -----

@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_pipeline_against_oracle(wid):
    """The step bench.py times, as separate calls: dedup -> K/V of the kept
    tokens -> head-aware -> compaction of hidden (merged), K and V; every
    sample, pruned row and slot against the oracle."""
    from paper_2608_25332_amd import provip
    w = workload(wid)
    dt = w.dtype
    _say(f"[pipeline-calls] workload {wid}")
    vis, anc = to_dev(w.vis, dt), to_dev(w.anchors, dt)
    q, kf, vf = to_dev(w.q, dt), to_dev(w.k_full, dt), to_dev(w.v_full, dt)
    r = provip.pv_prune_dedup(vis, anc, w.N1)
    k1, v1 = provip.pv_prune_gather_batch([kf, vf], r["kept"])
    h = provip.pv_prune_head_aware(q, k1, w.heads, w.N2)
    hid2, k2, v2 = provip.pv_prune_gather_batch([r["merged"], k1, v1], h["kept"])
    torch.cuda.synchronize()
    g = {k: to_host(r[k]) for k in ("kept", "score", "assign", "merged")}
    p_ref = oracle_p_workload(wid, w.anchors, w.vis)
    for b in range(w.spec.B):
        check_dedup_sample(g, b, w.vis[b], p_ref[b], w.N1, dt)
    kept1 = g["kept"]
    k1_ref = np.stack([w.k_full[b][:, kept1[b]] for b in range(w.spec.B)])
    assert np.array_equal(to_host(k1), k1_ref)
    _, v_ref = oracle.head_aware(w.q, k1_ref, w.heads, w.N2)
    kept2 = to_host(h["kept"])
    assert rel_err(to_host(h["score"]), v_ref) <= TOL[dt]
    for b in range(w.spec.B):
        check_kept(kept2[b], v_ref[b], w.N2, dt)
    assert np.array_equal(to_host(hid2), oracle.gather(g["merged"], kept2))
    assert np.array_equal(to_host(k2), oracle.gather(k1_ref, kept2))
    v1_ref = np.stack([w.v_full[b][:, kept1[b]] for b in range(w.spec.B)])
    assert np.array_equal(to_host(v2), oracle.gather(v1_ref, kept2))


def test_abi_errors_on_gpu():
    from paper_2608_25332_amd import provip
    x = torch.zeros((1, 64, 256), device="cuda:0")
    with pytest.raises(provip.ProvipError) as e:
        provip.pv_prune_dedup(x, x[:, :16], 65)
    assert e.value.status == -3
    q = torch.zeros((1, 4, 16, 64), device="cuda:0")
    with pytest.raises(provip.ProvipError) as e:
        provip.pv_prune_head_aware(q, q, [[1, 1]], 4)
    assert e.value.status == -4



@pytest.mark.parametrize("B,H,Nt,N,hd,nh", [(1, 4, 128, 960, 128, 4), (2, 6, 70, 1100, 64, 3)])
def test_head_aware_split_form_in_model(B, H, Nt, N, hd, nh):
    """The split score form on the model's softmax domain (row_lse merged
    after the chunks' statistics) and with a device head list, against the
    oracle."""
    from paper_2608_25332_amd import provip
    assert score_form(B, H, Nt, N, hd, nh, "bf16") == "split"
    rng = np.random.default_rng(B * 13 + N)
    q = W.bf16_round((rng.standard_normal((B, H, Nt, hd)) * 1.5).astype(np.float32))
    k = W.bf16_round((rng.standard_normal((B, H, N, hd)) * 1.5).astype(np.float32))
    heads = np.stack([rng.permutation(H)[:nh] for _ in range(B)]).astype(np.int32)
    ko = rng.standard_normal((B, H, 40, hd)) * 1.5
    lg = np.matmul(q.astype(np.float64), np.swapaxes(ko, -1, -2)) / np.sqrt(hd)
    mx = lg.max(-1, keepdims=True)
    lse = (mx[..., 0] + np.log(np.exp(lg - mx).sum(-1))).astype(np.float32)
    qd, kd = to_dev(q, "bf16"), to_dev(k, "bf16")
    r = provip.pv_prune_head_aware(qd, kd, heads, 100, row_lse=torch.from_numpy(lse).to("cuda:0"))
    r2 = provip.pv_prune_head_aware(qd, kd, torch.from_numpy(heads).to("cuda:0"), 100,
                                    row_lse=torch.from_numpy(lse).to("cuda:0"))
    torch.cuda.synchronize()
    assert torch.equal(r["score"], r2["score"]) and torch.equal(r["kept"], r2["kept"])
    v, kept = to_host(r["score"]), to_host(r["kept"])
    _, ref_v = oracle.head_aware_in_model(q, k, heads, lse.astype(np.float64), 100)
    assert rel_err(v, ref_v) <= TOL["bf16"], rel_err(v, ref_v)
    for b in range(B):
        check_kept(kept[b], ref_v[b], 100, "bf16")
