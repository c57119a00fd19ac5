"""Seeded synthetic inputs for the ProViP pruning hot path.

This module only draws inputs.  It contains none of the pruning arithmetic
(no cross-modal similarity, no centring, no attention, no selection), so the
HIP path and the CPU oracle can both be fed from it without sharing any of
the method's code.

Five workloads are defined, mirroring the shapes the paper evaluates on
(LLaVA-1.5-7B: 576 visual tokens, 4096 hidden, 32 heads x 128; LLaVA-NeXT
AnyRes: up to 5 x 576 tokens; a 13B-width backbone: 5120 hidden, 40 heads),
see the appendix "VLM Models" and Table "Efficiency".  The paper's images,
prompts and weights are not used: every tensor here is drawn from a seeded
Gaussian recipe, stated per workload below.

Every tensor gets its own random stream via ``SeedSequence(seed).spawn``.
Values are drawn in float32 and rounded once to bfloat16 with
round-to-nearest-even (workload 1 stays float32).  For bfloat16 workloads the
arrays returned are the exact float32 values of the bf16 numbers together
with the raw 16-bit patterns, so both paths read identical inputs.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import numpy as np

__all__ = [
    "WORKLOADS",
    "Workload",
    "make_workload",
    "bf16_round",
    "bf16_bits",
    "bf16_from_bits",
]


# --------------------------------------------------------------------------
# bfloat16 helpers (input marshalling only)
# --------------------------------------------------------------------------

def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even) and return
    the 16-bit patterns as uint16.  Inputs must be finite."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if not np.all(np.isfinite(x)):
        raise ValueError("bf16_bits: non-finite input")
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_from_bits(bits: np.ndarray) -> np.ndarray:
    """Exact float32 values of bfloat16 bit patterns."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 -> nearest bfloat16 value (RNE), returned as float32."""
    return bf16_from_bits(bf16_bits(x))


# --------------------------------------------------------------------------
# Workload table
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Spec:
    wid: int
    name: str
    B: int
    Nv: int
    d: int
    H: int
    hd: int
    Nt: int
    n_heads: int
    N1: int
    N2: int
    dtype: str  # "f32" or "bf16"
    recipe: str


WORKLOADS: Dict[int, Spec] = {
    1: Spec(1, "tiny-fp32", B=1, Nv=64, d=256, H=4, hd=64, Nt=16, n_heads=1,
            N1=32, N2=16, dtype="f32",
            recipe="vis~N(0,1) with 8 planted exact-duplicate pairs; text, Q, K, V ~N(0,1); heads {1}"),
    2: Spec(2, "llava1.5-7b", B=1, Nv=576, d=4096, H=32, hd=128, Nt=64, n_heads=4,
            N1=192, N2=64, dtype="bf16",
            recipe="vis = N(0,1) + rank-8 spatially smooth field on a 24x24 grid (neighbour cos ~0.8); "
                   "Q/K/V = seeded Gaussian projections / sqrt(d)"),
    3: Spec(3, "llava1.5-7b-b16", B=16, Nv=576, d=4096, H=32, hd=128, Nt=64, n_heads=4,
            N1=192, N2=64, dtype="bf16",
            recipe="16 independent draws of the llava1.5-7b recipe, per-sample head subsets"),
    4: Spec(4, "llava-next-7b-hires", B=4, Nv=2880, d=4096, H=32, hd=128, Nt=128, n_heads=4,
            N1=960, N2=320, dtype="bf16",
            recipe="5 tiles x 576, each tile its own smooth field; ~10% of each tile are "
                   "near-duplicate followers (cos > 0.98) in clusters of 2-4"),
    5: Spec(5, "13b-8frame", B=2, Nv=4608, d=5120, H=40, hd=128, Nt=128, n_heads=5,
            N1=1152, N2=512, dtype="bf16",
            recipe="frame 0 like llava1.5-7b at d=5120; frames 1-7 = frame 0 + N(0, 0.1^2)"),
}


@dataclasses.dataclass
class Workload:
    """One seeded batch.  Float arrays hold exact values of the storage dtype
    (bf16 values widened to float32 for bf16 workloads)."""

    spec: Spec
    vis: np.ndarray        # [B, Nv, d]   visual embeddings (connector output)
    anchors: np.ndarray    # [B, Nt, d]   critical-text embeddings
    q: np.ndarray          # [B, H, Nt, hd] text-query rows at the pruning layer
    k_full: np.ndarray     # [B, H, Nv, hd] keys of all visual tokens
    v_full: np.ndarray     # [B, H, Nv, hd] values of all visual tokens
    heads: np.ndarray      # [B, n_heads] int32, distinct per sample
    N1: int
    N2: int
    dtype: str
    dup_pairs: Optional[np.ndarray] = None   # [n, 2] planted exact twins (a < b)
    followers: Optional[np.ndarray] = None   # [B, n, 2] (leader, follower) near-dups

    def bits(self, name: str) -> np.ndarray:
        """Raw uint16 bf16 patterns of a float array (bf16 workloads only)."""
        if self.dtype != "bf16":
            raise ValueError("bits() is only defined for bf16 workloads")
        return bf16_bits(getattr(self, name))


def _rng_streams(seed: int, n: int):
    return [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(n)]


def _smooth_fields(rng: np.random.Generator, rank: int, grid: int) -> np.ndarray:
    """rank x (grid*grid) spatial fields: sums of three 2-D cosines with at most
    two cycles per `grid` tokens and random phases (values over the grid)."""
    y, x = np.meshgrid(np.arange(grid), np.arange(grid), indexing="ij")
    out = np.zeros((rank, grid * grid), dtype=np.float64)
    for r in range(rank):
        f = np.zeros((grid, grid))
        for _ in range(3):
            ky, kx = rng.integers(0, 3, size=2)
            if ky == 0 and kx == 0:
                kx = 1
            phase = rng.uniform(0, 2 * math.pi)
            f += np.cos(2 * math.pi * (ky * y + kx * x) / grid + phase)
        out[r] = f.reshape(-1)
    return out


def _neighbour_pairs(grid: int) -> np.ndarray:
    idx = np.arange(grid * grid).reshape(grid, grid)
    right = np.stack([idx[:, :-1].reshape(-1), idx[:, 1:].reshape(-1)], 1)
    down = np.stack([idx[:-1, :].reshape(-1), idx[1:, :].reshape(-1)], 1)
    return np.concatenate([right, down], 0)


def _calibrate_scale(L: np.ndarray, d: int, pairs: np.ndarray, target: float) -> float:
    """Scale s such that the expected neighbour cosine of Z + s*L is `target`,
    with Z ~ N(0, I_d) independent of L (expected-value model: the noise adds
    d to each squared norm and nothing to a cross product)."""
    sq = np.einsum("nd,nd->n", L, L)
    cross = np.einsum("nd,nd->n", L[pairs[:, 0]], L[pairs[:, 1]])

    def mean_cos(s):
        s2 = s * s
        return float(np.mean(s2 * cross / np.sqrt((d + s2 * sq[pairs[:, 0]]) * (d + s2 * sq[pairs[:, 1]]))))

    lo, hi = 0.0, 1.0
    while mean_cos(hi) < target:
        hi *= 2.0
        if hi > 1e6:
            raise RuntimeError("smooth field too rough to reach the target neighbour cosine")
    for _ in range(80):
        mid = 0.5 * (lo + hi)
        if mean_cos(mid) < target:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def _smooth_tile(rng: np.random.Generator, d: int, grid: int = 24, rank: int = 8,
                 target_cos: float = 0.80) -> np.ndarray:
    """grid*grid visual tokens: N(0,1) noise plus a calibrated rank-`rank`
    spatially smooth component.  float64 [grid*grid, d]."""
    fields = _smooth_fields(rng, rank, grid)                    # [rank, n]
    u = rng.standard_normal((rank, d))                          # [rank, d]
    L = fields.T @ u                                            # [n, d]
    s = _calibrate_scale(L, d, _neighbour_pairs(grid), target_cos)
    Z = rng.standard_normal((grid * grid, d))
    return Z + s * L


def _project_heads(x: np.ndarray, w: np.ndarray, H: int, hd: int) -> np.ndarray:
    """x [n, d] @ w [d, H*hd] -> [H, n, hd] (float32 matmul)."""
    y = x.astype(np.float32) @ w
    return np.ascontiguousarray(y.reshape(x.shape[0], H, hd).transpose(1, 0, 2))


def make_workload(wid: int, seed: Optional[int] = None, *, B: Optional[int] = None,
                  with_kv: bool = True) -> Workload:
    """Draw workload `wid` (1..5) with `seed` (default: the workload number).

    ``B`` overrides the batch size (each sample is an independent draw of the
    same recipe).  ``with_kv=False`` skips the key/value projections of the
    visual tokens (the most expensive part of the draw) and leaves
    ``k_full``/``v_full`` empty."""
    spec = WORKLOADS[wid]
    if B is not None:
        spec = dataclasses.replace(spec, B=int(B))
    seed = wid if seed is None else int(seed)
    st = _rng_streams(seed, 8)
    rng_vis, rng_txt, rng_w, rng_heads, rng_dup, rng_q, rng_kv, _ = st
    Bn, Nv, d, H, hd, Nt = spec.B, spec.Nv, spec.d, spec.H, spec.hd, spec.Nt

    dup_pairs = None
    followers = None
    if wid == 1:
        vis = rng_vis.standard_normal((Bn, Nv, d)).astype(np.float32)
        perm = rng_dup.permutation(Nv)[:16].reshape(8, 2)
        dup_pairs = np.sort(perm, axis=1).astype(np.int64)
        for a, b in dup_pairs:
            vis[:, b] = vis[:, a]
        anchors = rng_txt.standard_normal((Bn, Nt, d)).astype(np.float32)
        q = rng_q.standard_normal((Bn, H, Nt, hd)).astype(np.float32)
        if with_kv:
            k_full = rng_kv.standard_normal((Bn, H, Nv, hd)).astype(np.float32)
            v_full = rng_kv.standard_normal((Bn, H, Nv, hd)).astype(np.float32)
        else:
            k_full = v_full = np.zeros((Bn, H, 0, hd), np.float32)
        heads = np.ones((Bn, 1), dtype=np.int32)
        return Workload(spec, vis, anchors, q, k_full, v_full, heads, spec.N1, spec.N2,
                        spec.dtype, dup_pairs=dup_pairs)

    # bf16 workloads
    vis = np.empty((Bn, Nv, d), dtype=np.float32)
    fol = []
    for b in range(Bn):
        if wid in (2, 3):
            vis[b] = _smooth_tile(rng_vis, d)
        elif wid == 4:
            tiles = []
            fb = []
            for t in range(Nv // 576):
                tile = _smooth_tile(rng_vis, d)
                # near-duplicate clusters: ~10% of the tile are followers of a leader
                order = rng_dup.permutation(576)
                n_fol, pos = 0, 0
                while n_fol < 58:
                    size = int(rng_dup.integers(2, 5))          # cluster of 2..4
                    size = min(size, 58 - n_fol + 1)
                    leader = order[pos]
                    members = order[pos + 1: pos + size]
                    pos += size
                    lnorm = np.linalg.norm(tile[leader])
                    eps = 0.1 * lnorm / math.sqrt(d)
                    for m in members:
                        tile[m] = tile[leader] + eps * rng_dup.standard_normal(d)
                        fb.append((t * 576 + leader, t * 576 + m))
                    n_fol += len(members)
                tiles.append(tile)
            vis[b] = np.concatenate(tiles, 0)
            fol.append(np.array(fb, dtype=np.int64))
        elif wid == 5:
            f0 = _smooth_tile(rng_vis, d)
            frames = [f0] + [f0 + 0.1 * rng_vis.standard_normal(f0.shape) for _ in range(7)]
            vis[b] = np.concatenate(frames, 0)
        else:
            raise ValueError(wid)
    if fol:
        n = min(len(f) for f in fol)
        followers = np.stack([f[:n] for f in fol], 0)
    vis = bf16_round(vis)
    text = rng_txt.standard_normal((Bn, Nt, d)).astype(np.float32)
    anchors = bf16_round(text)

    scale = 1.0 / math.sqrt(d)
    wq = (rng_w.standard_normal((d, H * hd), dtype=np.float32) * np.float32(scale))
    q = np.stack([_project_heads(text[b], wq, H, hd) for b in range(Bn)], 0)
    q = bf16_round(q)
    del wq
    if with_kv:
        wk = (rng_w.standard_normal((d, H * hd), dtype=np.float32) * np.float32(scale))
        k_full = bf16_round(np.stack([_project_heads(vis[b], wk, H, hd) for b in range(Bn)], 0))
        del wk
        wv = (rng_w.standard_normal((d, H * hd), dtype=np.float32) * np.float32(scale))
        v_full = bf16_round(np.stack([_project_heads(vis[b], wv, H, hd) for b in range(Bn)], 0))
        del wv
    else:
        k_full = v_full = np.zeros((Bn, H, 0, hd), np.float32)
    heads = np.stack([np.sort(rng_heads.permutation(H)[:spec.n_heads]) for _ in range(Bn)], 0)
    heads = heads.astype(np.int32)
    return Workload(spec, vis, anchors, q, k_full, v_full, heads, spec.N1, spec.N2, spec.dtype,
                    dup_pairs=dup_pairs, followers=followers)


def make_middle_layer(w: Workload, seed: Optional[int] = None):
    """Text-query rows and keys of every visual token at a second, deeper
    pruning layer, for the progressive schedule: the first layer's recipe
    with projections of their own (seeded by `seed`, default 1000 + the
    workload number).  Returns (q_m [B,H,Nt,hd], k_m_all [B,H,Nv,hd]) in the
    workload's storage values (bf16 values widened to float32, or float32)."""
    s = w.spec
    seed = 1000 + s.wid if seed is None else int(seed)
    rng_q, rng_k = _rng_streams(seed, 2)
    Bn, Nv, d, H, hd, Nt = s.B, s.Nv, s.d, s.H, s.hd, s.Nt
    if w.dtype == "f32":
        q = rng_q.standard_normal((Bn, H, Nt, hd)).astype(np.float32)
        k = rng_k.standard_normal((Bn, H, Nv, hd)).astype(np.float32)
        return q, k
    scale = np.float32(1.0 / math.sqrt(d))
    wq = rng_q.standard_normal((d, H * hd), dtype=np.float32) * scale
    q = bf16_round(np.stack([_project_heads(w.anchors[b], wq, H, hd) for b in range(Bn)], 0))
    del wq
    wk = rng_k.standard_normal((d, H * hd), dtype=np.float32) * scale
    k = bf16_round(np.stack([_project_heads(w.vis[b], wk, H, hd) for b in range(Bn)], 0))
    return q, k


def progressive_budgets(spec: Spec):
    """Budgets of the progressive schedule for a workload: N1 and N2 of the
    workload, N3 = N2 / 2 at the middle layer, and N_vis = 6 visual heads
    (the paper's setting; half the heads where there are fewer than 12)."""
    return spec.N1, min(6, spec.H // 2), spec.N2, max(1, spec.N2 // 2)
