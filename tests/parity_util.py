"""Helpers shared by the GPU parity tests: device marshalling of the seeded
inputs and the comparison rules (tolerances, near-tie exemptions)."""

from __future__ import annotations

import numpy as np

from paper_2608_25332_amd import workloads as W

# max |gpu - oracle| / max |oracle| for float outputs
TOL = {"f32": 1e-5, "bf16": 2e-3}
# selection decisions closer than this (relative to max |score|) to the k-th
# value may go either way; those tokens are exempt from the bit-exact check
TAU = {"f32": 1e-6, "bf16": 1e-4}
# nearest-centroid decisions with a top-2 cosine gap below this are exempt
TAU_ASSIGN = {"f32": 1e-6, "bf16": 1e-4}


def to_dev(arr: np.ndarray, dtype: str, device="cuda:0"):
    import torch

    if dtype == "bf16":
        bits = W.bf16_bits(np.asarray(arr, np.float32))
        t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32))
    return t.to(device)


def to_host(t) -> np.ndarray:
    import torch

    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy()
    return t.cpu().numpy()


def rel_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    den = float(np.max(np.abs(ref)))
    if den == 0.0:
        den = 1.0
    return float(np.max(np.abs(np.asarray(gpu, np.float64) - ref))) / den


def check_kept(gpu_kept: np.ndarray, score_ref: np.ndarray, k: int, dtype: str):
    """Kept set must equal the oracle's, except tokens whose oracle score lies
    within TAU of the k-th largest oracle score.  Returns #exempt tokens."""
    import oracle

    g = np.asarray(gpu_kept)
    assert g.shape == (k,)
    assert np.all(np.diff(g) > 0), "kept indices must be strictly increasing"
    assert g.min() >= 0 and g.max() < score_ref.shape[0]
    ref = oracle.topk(score_ref, k)
    kth = np.sort(score_ref)[::-1][k - 1]
    tau = TAU[dtype] * max(float(np.max(np.abs(score_ref))), 1e-30)
    exempt = set(np.nonzero(np.abs(score_ref - kth) <= tau)[0].tolist())
    a = set(g.tolist()) - exempt
    b = set(ref.tolist()) - exempt
    assert a == b, f"kept differs outside the near-tie band: +{sorted(a - b)[:8]} -{sorted(b - a)[:8]}"
    return len(exempt)


def check_assign_rows(gpu_assign: np.ndarray, vis: np.ndarray, kept: np.ndarray, rows,
                      dtype: str):
    """Oracle nearest centroid (with the GPU's kept list) for `rows`; must
    match bit for bit except rows whose top-2 cosine gap is below TAU_ASSIGN.
    Returns #exempt rows."""
    import oracle

    rows = np.asarray(rows, np.int32)
    a, b1, b2 = oracle.assign(vis, kept, rows)
    g = np.asarray(gpu_assign)[rows]
    close = (b1 - b2) < TAU_ASSIGN[dtype]
    bad = (g != a) & ~close
    assert not bad.any(), f"assign differs at rows {rows[bad][:8]}: gpu {g[bad][:8]} oracle {a[bad][:8]}"
    return int(close.sum())


def check_merged(gpu_merged: np.ndarray, vis: np.ndarray, kept, assign, slots, dtype: str):
    """Oracle merge (given the GPU's kept/assign) for the listed slots."""
    import oracle

    ref = oracle.merge(vis, kept, assign)[slots]
    g = np.asarray(gpu_merged, np.float64)[slots]
    if dtype == "bf16":
        r = W.bf16_round(ref.astype(np.float32)).astype(np.float64)
        # at most one bf16 ulp from the correctly rounded mean
        ulp = np.maximum(np.abs(r), np.abs(g)) * 2.0 ** -7 + 1e-38
        assert np.all(np.abs(g - r) <= ulp * 1.0001), float(np.max(np.abs(g - r) / ulp))
    else:
        assert rel_err(g, ref) <= TOL["f32"]


from oracle.parallel import oracle_assign, oracle_p, workers  # noqa: E402,F401


def check_assign_all(gpu_assign: np.ndarray, vis_b: np.ndarray, kept: np.ndarray, dtype: str):
    """check_assign_rows over every pruned row of one sample, with the oracle
    run in parallel.  Returns #exempt rows."""
    pruned = np.setdiff1d(np.arange(vis_b.shape[0]), kept).astype(np.int32)
    if len(pruned) == 0:
        return 0
    a, b1, b2 = oracle_assign(vis_b, kept, pruned)
    g = np.asarray(gpu_assign)[pruned]
    close = (b1 - b2) < TAU_ASSIGN[dtype]
    bad = (g != a) & ~close
    assert not bad.any(), (f"assign differs at rows {pruned[bad][:8]}: gpu {g[bad][:8]} "
                           f"oracle {a[bad][:8]}")
    return int(close.sum())


def check_dedup_sample(g: dict, b: int, vis_b: np.ndarray, p_ref: np.ndarray, n1: int,
                       dtype: str):
    """One sample of pv_prune_dedup's outputs (keys kept/score/assign/merged,
    host arrays) against the oracle: p, the kept set, the nearest kept token
    of every pruned row and every merged slot.  Returns (#near-tie tokens,
    #near-tie rows)."""
    assert rel_err(g["score"][b], p_ref) <= TOL[dtype], rel_err(g["score"][b], p_ref)
    kept = np.asarray(g["kept"][b])
    ex_k = check_kept(kept, p_ref, n1, dtype)
    ex_a = check_assign_all(g["assign"][b], vis_b, kept, dtype)
    check_merged(g["merged"][b], vis_b, kept, g["assign"][b], np.arange(n1), dtype)
    return ex_k, ex_a


_P_CACHE: dict = {}


def oracle_p_workload(wid: int, anchors: np.ndarray, vis: np.ndarray) -> np.ndarray:
    """oracle_p of a seeded workload, computed once per process."""
    if wid not in _P_CACHE:
        _P_CACHE[wid] = oracle_p(anchors, vis)
    return _P_CACHE[wid]
