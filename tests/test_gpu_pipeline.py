"""The whole pruning step in one call (pv_prune_pipeline).

Where the shapes allow it, the two chains that follow the top-N_1 selection
share launches (the score, on the kept tokens' keys read through the kept
list, rides with the Gram tiles; the top-N_2, the Gram's argmax and the K/V
compaction share the next launch; the merge writes the kept slots' hidden
rows and carries the final K/V compaction).  Every output
must equal, bit for bit, the same step with every kernel in its own launch
(pv_prune_pipeline_separate, which is the four calls made one after another),
and the step must match the oracle as the separate calls do.
"""

from __future__ import annotations

import functools
import sys

import numpy as np
import pytest

import oracle
from paper_2608_25332_amd import workloads as W
from parity_util import (TOL, check_dedup_sample, check_kept, oracle_p_workload, rel_err, to_dev,
                         to_host)

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
def workload(wid: int):
    return W.make_workload(wid)


def _inputs(w):
    dt = w.dtype
    return (to_dev(w.vis, dt), to_dev(w.anchors, dt), to_dev(w.q, dt), to_dev(w.k_full, dt),
            to_dev(w.v_full, dt))


def _both(ins, heads, N1, N2):
    """Outputs of the shared-launch step and of the separate step, each into
    buffers filled with a different pattern first (so that nothing left in
    place by one passes for the other's result)."""
    from paper_2608_25332_amd import provip
    res = []
    for sep, fill in ((False, 0x5A), (True, 0x3C)):
        o = provip.pv_prune_pipeline(*ins, heads, N1, N2, separate=sep)
        for n in provip.PIPELINE_OUTPUTS:
            o[n].view(torch.uint8).fill_(fill)
        o = provip.pv_prune_pipeline(*ins, heads, N1, N2, out=o, workspace=o["workspace"],
                                     separate=sep)
        torch.cuda.synchronize()
        res.append(o)
    return res


def _assert_same(a, b):
    from paper_2608_25332_amd import provip
    for n in provip.PIPELINE_OUTPUTS:
        x = a[n].view(torch.uint8) if a[n].dtype == torch.bfloat16 else a[n]
        y = b[n].view(torch.uint8) if b[n].dtype == torch.bfloat16 else b[n]
        assert torch.equal(x, y), f"{n} differs between the shared and the separate launches"


@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_pipeline_shared_launches_equal_separate(wid):
    w = workload(wid)
    _say(f"[pipeline] workload {wid} ({w.spec.name})")
    fused, sep = _both(_inputs(w), w.heads, w.N1, w.N2)
    _assert_same(fused, sep)


@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_pipeline_against_oracle(wid):
    """The step bench.py times, in one call, against the oracle: every
    sample's p and kept set, the nearest kept token of every pruned row,
    every merged slot, the head-aware score and selection, and the
    compacted tensors byte for byte."""
    from paper_2608_25332_amd import provip
    w = workload(wid)
    dt = w.dtype
    _say(f"[pipeline-oracle] workload {wid}")
    o = provip.pv_prune_pipeline(*_inputs(w), w.heads, w.N1, w.N2)
    torch.cuda.synchronize()
    g = {"kept": to_host(o["kept1"]), "score": to_host(o["score1"]),
         "assign": to_host(o["assign"]), "merged": to_host(o["merged"])}
    p_ref = oracle_p_workload(wid, w.anchors, w.vis)
    for b in range(w.spec.B):
        check_dedup_sample(g, b, w.vis[b], p_ref[b], w.N1, dt)
    kept1 = g["kept"]
    k1_ref = np.stack([w.k_full[b][:, kept1[b]] for b in range(w.spec.B)])
    v1_ref = np.stack([w.v_full[b][:, kept1[b]] for b in range(w.spec.B)])
    assert np.array_equal(to_host(o["k1"]), k1_ref)
    assert np.array_equal(to_host(o["v1"]), v1_ref)
    _, v_ref = oracle.head_aware(w.q, k1_ref, w.heads, w.N2)
    assert rel_err(to_host(o["score2"]), v_ref) <= TOL[dt]
    kept2 = to_host(o["kept2"])
    for b in range(w.spec.B):
        check_kept(kept2[b], v_ref[b], w.N2, dt)
    assert np.array_equal(to_host(o["hidden2"]), oracle.gather(g["merged"], kept2))
    assert np.array_equal(to_host(o["k2"]), oracle.gather(k1_ref, kept2))
    assert np.array_equal(to_host(o["v2"]), oracle.gather(v1_ref, kept2))
    if wid == 1:
        # the tiny fp32 workload has no near ties: the whole step is exact
        ref = oracle.dedup(w.anchors, w.vis, w.N1)
        assert np.array_equal(g["kept"], ref["kept"])
        assert np.array_equal(g["assign"], ref["assign"])
        assert np.max(np.abs(g["merged"] - ref["merged"])) <= 1e-5 * np.max(np.abs(ref["merged"]))


# (B, Nv, Nt, d, H, hd, n_heads, N1, N2, dtype, shared): shapes on both sides
# of every condition for the shared launches (split-k Gram; 16-row score
# blocks over 256-byte head rows; the plain merge - one sample with
# N1 x ceil(row bytes / 1 KiB) x 4 <= row bytes -; N1 <= 256); `shared` says
# whether the step must take them
EDGE = [
    (1, 100, 5, 512, 2, 128, 1, 37, 5, "bf16", True),       # ragged tiles, one head
    (1, 300, 20, 512, 8, 128, 3, 256, 100, "bf16", True),   # N1 = 256: the widest carried top-k (four key chunks)
    (1, 300, 20, 512, 8, 128, 3, 257, 100, "bf16", False),  # N1 = 257: member-list merge
    (1, 300, 20, 512, 8, 128, 3, 100, 30, "bf16", True),    # two key chunks in the shared score
    (1, 300, 20, 512, 8, 128, 3, 100, 100, "bf16", True),   # N2 = N1: every slot's row compacted
    (1, 130, 7, 512, 8, 128, 8, 65, 64, "bf16", True),      # 65 keys: one past a chunk, all heads
    (1, 64, 16, 512, 4, 64, 2, 64, 10, "bf16", False),      # N1 = Nv: nothing pruned, no Gram
    (1, 90, 16, 512, 4, 64, 2, 40, 7, "bf16", False),       # 128-byte head rows
    (1, 90, 16, 256, 4, 64, 2, 40, 7, "f32", True),         # 256-byte fp32 head rows
    (1, 500, 130, 512, 8, 128, 4, 200, 50, "bf16", True),   # nine 16-row score blocks
    (1, 1500, 100, 512, 8, 128, 4, 250, 60, "bf16", True),  # many pruned rows
    (1, 1500, 20, 2048, 8, 128, 2, 250, 60, "bf16", False),  # wide split-k Gram tiles
    (1, 40, 3, 64, 1, 128, 1, 1, 1, "bf16", True),          # budgets of one
    (1, 200, 8, 64, 2, 128, 2, 100, 9, "bf16", False),      # member-list merge (narrow rows)
    (1, 1300, 16, 64, 2, 128, 1, 1024, 50, "bf16", False),  # N1 = 1024
    (2, 90, 16, 256, 4, 64, 2, 40, 7, "f32", False),        # two samples: member-list merge
    (65, 100, 80, 64, 8, 128, 8, 40, 10, "bf16", False),    # 520 head pairs: two score launches
    (8, 576, 64, 512, 8, 128, 4, 192, 64, "bf16", False),   # LLaVA-like token counts, batch
    (8, 2000, 16, 64, 2, 128, 1, 600, 50, "bf16", False),   # full-k Gram tiles
    (32, 100, 16, 64, 8, 128, 4, 50, 10, "bf16", False),    # whole-head score form
    (1, 300, 20, 520, 8, 80, 3, 100, 30, "bf16", False),    # padded widths: separate launches
    (2, 150, 10, 72, 4, 40, 2, 60, 12, "f32", False),
]


@pytest.mark.parametrize("B,Nv,Nt,d,H,hd,nh,N1,N2,dt,shared", EDGE)
def test_pipeline_edges(B, Nv, Nt, d, H, hd, nh, N1, N2, dt, shared):
    from paper_2608_25332_amd import provip
    _say(f"[pipeline-edge] B={B} Nv={Nv} Nt={Nt} d={d} H={H} hd={hd} heads={nh} "
         f"N1={N1} N2={N2} {dt}")
    rng = np.random.default_rng(B * 1000 + Nv + N1)
    f = (lambda a: W.bf16_round(a)) if dt == "bf16" else (lambda a: a)
    vis = f(rng.standard_normal((B, Nv, d)).astype(np.float32))
    anc = f(rng.standard_normal((B, Nt, d)).astype(np.float32))
    q = f(rng.standard_normal((B, H, Nt, hd)).astype(np.float32))
    kf = f(rng.standard_normal((B, H, Nv, hd)).astype(np.float32))
    vf = f(rng.standard_normal((B, H, Nv, hd)).astype(np.float32))
    heads = np.stack([rng.permutation(H)[:nh] for _ in range(B)]).astype(np.int32)
    ins = tuple(to_dev(a, dt) for a in (vis, anc, q, kf, vf))
    fused, sep = _both(ins, heads, N1, N2)
    _assert_same(fused, sep)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(10)]
    for e in ev:
        e.record()
    timed = provip.pv_prune_pipeline(*ins, heads, N1, N2, events=ev)
    torch.cuda.synchronize()
    assert (timed["n_kernels"] > 0) == shared, timed.get("kernel_names")
    _assert_same(timed, sep)
    # the separate step is the four calls: every sample against the oracle
    # (p, kept set, the nearest kept token of every pruned row, every merged
    # slot, the head-aware score and selection)
    sh = {"kept": to_host(sep["kept1"]), "score": to_host(sep["score1"]),
          "assign": to_host(sep["assign"]), "merged": to_host(sep["merged"])}
    for b in range(B):
        ref = oracle.dedup(anc[b:b + 1], vis[b:b + 1], N1, want_assign=False)
        check_dedup_sample(sh, b, vis[b], ref["p"][0], N1, dt)
        kept1 = sh["kept"][b]
        _, v_ref = oracle.head_aware(q[b:b + 1], kf[b:b + 1][:, :, kept1], heads[b:b + 1], N2)
        assert rel_err(to_host(sep["score2"])[b], v_ref[0]) <= TOL[dt]
        check_kept(to_host(sep["kept2"])[b], v_ref[0], N2, dt)


@pytest.mark.parametrize("wid", [2, 3])
def test_pipeline_timed_reps_leave_results_unchanged(wid):
    """The timed call (events around each launch, every launch repeated)
    gives the untimed call's outputs and names the shared launches."""
    from paper_2608_25332_amd import provip
    w = workload(wid)
    _say(f"[pipeline-timed] workload {wid}")
    ins = _inputs(w)
    ref = provip.pv_prune_pipeline(*ins, w.heads, w.N1, w.N2)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(10)]
    for e in ev:
        e.record()
    got = provip.pv_prune_pipeline(*ins, w.heads, w.N1, w.N2, events=ev, reps=3)
    torch.cuda.synchronize()
    _assert_same(got, ref)
    if wid == 2:
        assert got["kernel_names"] == ["cos_full", "center", "select",
                                       "gram_partial+score_partial",
                                       "gram_reduce+score_select+gather_kv1",
                                       "merge+gather_hkv2"]
    else:  # B = 16: member-list merge, separate launches
        assert got["n_kernels"] == 0
