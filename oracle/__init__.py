"""CPU oracle for ProViP's pruning hot path (test infrastructure).

This package is the slow, plain reference the HIP path is checked against.
Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import it; the product package never does.  It shares no
code with the HIP library: the arithmetic lives in ``provip_oracle.c``
(fp64, plain loops) and this module only marshals numpy arrays through
ctypes, one sample at a time.

Function map (paper passages are cited at each C function):
  critical_text              -- Sec. 4.2, equations for r and T
  cosine / center / maxpool  -- Sec. 4.3, equations for M, M-hat and p
  topk                       -- retention of the N_1 / N_2 highest scores
  assign / merge             -- Sec. 4.3, nearest-centroid aggregation
  attention / head_aware     -- Sec. 4.4, equations for S^vis and v
  attention_in_model /
  head_aware_in_model        -- Sec. 4.4 on the visual slice of the model's softmax
  head_confidence /
  visual_heads               -- Sec. 4.4, equations for C^h and V_l
  head_confidence_in_model /
  visual_heads_in_model      -- the same on the visual slice of the model's softmax
  gather                     -- compaction of kept rows (Sec. 4.1)
  dedup                      -- Sec. 4.3 end to end

parity unpinned: ``merge`` (the paper names no aggregation formula).
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "provip_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(out_path: str = _LIB_PATH, src_path: str = _SRC) -> str:
    """Compile the oracle with gcc (IEEE fp64, no fast-math)."""
    cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fno-fast-math",
           "-o", out_path, src_path, "-lm"]
    subprocess.run(cmd, check=True)
    return out_path


def load(path: str = _LIB_PATH, *, rebuild_if_missing: bool = True):
    """Load (building once if nothing is built) and return the ctypes handle."""
    global _lib
    if _lib is not None and path == _LIB_PATH:
        return _lib
    if not os.path.exists(path):
        if not rebuild_if_missing:
            raise FileNotFoundError(path)
        build(path)
    lib = ctypes.CDLL(path)
    _declare(lib)
    if path == _LIB_PATH:
        _lib = lib
    return lib


_D = ctypes.POINTER(ctypes.c_double)
_I = ctypes.POINTER(ctypes.c_int32)
_U8 = ctypes.POINTER(ctypes.c_uint8)
_int = ctypes.c_int
_i64 = ctypes.c_int64


def _declare(lib):
    lib.orc_cosine.argtypes = [_D, _int, _D, _int, _int, _D]
    lib.orc_cosine.restype = None
    lib.orc_center.argtypes = [_D, _int, _int, _D]
    lib.orc_center.restype = None
    lib.orc_maxpool.argtypes = [_D, _int, _int, _D]
    lib.orc_maxpool.restype = None
    lib.orc_topk.argtypes = [_D, _int, _int, _I]
    lib.orc_topk.restype = _int
    lib.orc_assign.argtypes = [_D, _int, _int, _I, _int, _I, _int, _I, _D, _D]
    lib.orc_assign.restype = None
    lib.orc_merge.argtypes = [_D, _int, _int, _I, _int, _I, _D]
    lib.orc_merge.restype = None
    lib.orc_dedup.argtypes = [_D, _int, _D, _int, _int, _int, _I, _D, _I, _D]
    lib.orc_dedup.restype = _int
    lib.orc_attention.argtypes = [_D, _D, _int, _int, _int, _D]
    lib.orc_attention.restype = None
    lib.orc_head_aware_score.argtypes = [_D, _D, _int, _int, _int, _int, _I, _int, _D]
    lib.orc_head_aware_score.restype = _int
    lib.orc_head_aware.argtypes = [_D, _D, _int, _int, _int, _int, _I, _int, _int, _I, _D]
    lib.orc_head_aware.restype = _int
    lib.orc_critical_text.argtypes = [_D, _int, _int, _D, _I]
    lib.orc_critical_text.restype = _int
    lib.orc_attention_in_model.argtypes = [_D, _D, _D, _int, _int, _int, _D]
    lib.orc_attention_in_model.restype = None
    lib.orc_head_aware_score_in_model.argtypes = [_D, _D, _D, _int, _int, _int, _int, _I, _int, _D]
    lib.orc_head_aware_score_in_model.restype = _int
    lib.orc_head_confidence.argtypes = [_D, _D, _int, _int, _int, _int, _D]
    lib.orc_head_confidence.restype = _int
    lib.orc_visual_heads.argtypes = [_D, _D, _int, _int, _int, _int, _int, _I, _D]
    lib.orc_visual_heads.restype = _int
    lib.orc_head_confidence_in_model.argtypes = [_D, _D, _D, _int, _int, _int, _int, _D]
    lib.orc_head_confidence_in_model.restype = _int
    lib.orc_visual_heads_in_model.argtypes = [_D, _D, _D, _int, _int, _int, _int, _int, _I, _D]
    lib.orc_visual_heads_in_model.restype = _int
    lib.orc_gather.argtypes = [_U8, _U8, _I, _int, _int, _int, _int, _i64,
                               _i64, _i64, _i64, _i64, _i64, _i64]
    lib.orc_gather.restype = _int


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _pd(a: np.ndarray):
    return a.ctypes.data_as(_D)


def _pi(a: np.ndarray):
    return a.ctypes.data_as(_I)


class OracleError(RuntimeError):
    pass


# ------------------------------------------------------- critical text --

def critical_text(text, *, lib=None):
    """Sec. 4.2 over a batch: text [B, nt, d] -> (r [B, nt], mask [B, nt]
    int32 with 1 for the critical tokens, count [B])."""
    lib = lib or load()
    E = _f64(text)
    B, nt, d = E.shape
    r = np.empty((B, nt), np.float64)
    mask = np.empty((B, nt), np.int32)
    count = np.empty(B, np.int32)
    for b in range(B):
        c = lib.orc_critical_text(_pd(E[b]), nt, d, _pd(r[b]), _pi(mask[b]))
        if c < 0:
            raise OracleError(f"orc_critical_text rc={c}")
        count[b] = c
    return r, mask, count


# ---------------------------------------------------------------- stage A --

def cosine(anchors, vis, *, lib=None) -> np.ndarray:
    """M for one sample: anchors [nt, d], vis [nv, d] -> [nt, nv]."""
    lib = lib or load()
    a, v = _f64(anchors), _f64(vis)
    nt, d = a.shape
    nv = v.shape[0]
    M = np.empty((nt, nv), np.float64)
    lib.orc_cosine(_pd(a), nt, _pd(v), nv, d, _pd(M))
    return M


def center(M, *, lib=None) -> np.ndarray:
    lib = lib or load()
    M = _f64(M)
    out = np.empty_like(M)
    lib.orc_center(_pd(M), M.shape[0], M.shape[1], _pd(out))
    return out


def maxpool(Mhat, *, lib=None) -> np.ndarray:
    lib = lib or load()
    Mh = _f64(Mhat)
    p = np.empty(Mh.shape[1], np.float64)
    lib.orc_maxpool(_pd(Mh), Mh.shape[0], Mh.shape[1], _pd(p))
    return p


def topk(score, k: int, *, lib=None) -> np.ndarray:
    """Top-k of a 1-D score vector, lowest index wins ties, ascending output."""
    lib = lib or load()
    s = _f64(score)
    out = np.empty(int(k), np.int32)
    rc = lib.orc_topk(_pd(s), s.shape[0], int(k), _pi(out))
    if rc != 0:
        raise OracleError(f"orc_topk rc={rc}")
    return out


def assign(vis, kept, rows: Optional[Sequence[int]] = None, *, lib=None):
    """Nearest-centroid slot per row (all tokens when rows is None).
    Returns (assign, best_cos, second_cos)."""
    lib = lib or load()
    v = _f64(vis)
    kp = _i32(kept)
    nv, d = v.shape
    if rows is None:
        r = None
        n = nv
    else:
        r = _i32(rows)
        n = r.shape[0]
    a = np.empty(n, np.int32)
    b1 = np.empty(n, np.float64)
    b2 = np.empty(n, np.float64)
    lib.orc_assign(_pd(v), nv, d, _pi(kp), kp.shape[0], _pi(r) if r is not None else None,
                   n, _pi(a), _pd(b1), _pd(b2))
    return a, b1, b2


def merge(vis, kept, assign_, *, lib=None) -> np.ndarray:
    lib = lib or load()
    v = _f64(vis)
    kp = _i32(kept)
    a = _i32(assign_)
    nv, d = v.shape
    out = np.empty((kp.shape[0], d), np.float64)
    lib.orc_merge(_pd(v), nv, d, _pi(kp), kp.shape[0], _pi(a), _pd(out))
    return out


def dedup(anchors, vis, n1: int, *, want_assign: bool = True, lib=None):
    """Sec. 4.3 end to end over a batch.
    anchors [B, nt, d], vis [B, nv, d] -> dict(kept [B,n1], p [B,nv],
    assign [B,nv], merged [B,n1,d]) (assign/merged only if want_assign)."""
    lib = lib or load()
    A, V = _f64(anchors), _f64(vis)
    B, nt, d = A.shape
    nv = V.shape[1]
    kept = np.empty((B, n1), np.int32)
    p = np.empty((B, nv), np.float64)
    asg = np.empty((B, nv), np.int32) if want_assign else None
    mrg = np.empty((B, n1, d), np.float64) if want_assign else None
    for b in range(B):
        rc = lib.orc_dedup(_pd(A[b]), nt, _pd(V[b]), nv, d, int(n1), _pi(kept[b]), _pd(p[b]),
                           _pi(asg[b]) if want_assign else None,
                           _pd(mrg[b]) if want_assign else None)
        if rc != 0:
            raise OracleError(f"orc_dedup rc={rc}")
    return {"kept": kept, "p": p, "assign": asg, "merged": mrg}


# ---------------------------------------------------------------- stage B --

def attention(q, k, *, lib=None) -> np.ndarray:
    """One head: q [nt, hd], k [n, hd] -> softmax(q k^T / sqrt(hd)) [nt, n]."""
    lib = lib or load()
    q, k = _f64(q), _f64(k)
    nt, hd = q.shape
    n = k.shape[0]
    A = np.empty((nt, n), np.float64)
    lib.orc_attention(_pd(q), _pd(k), nt, n, hd, _pd(A))
    return A


def head_aware_score(q, k, heads, *, lib=None) -> np.ndarray:
    """One sample: q [H, nt, hd], k [H, n, hd], heads list -> v [n]."""
    lib = lib or load()
    q, k = _f64(q), _f64(k)
    hs = _i32(heads)
    H, nt, hd = q.shape
    n = k.shape[1]
    v = np.empty(n, np.float64)
    rc = lib.orc_head_aware_score(_pd(q), _pd(k), H, nt, n, hd, _pi(hs), hs.shape[0], _pd(v))
    if rc != 0:
        raise OracleError(f"orc_head_aware_score rc={rc}")
    return v


def head_aware(q, k, heads, n2: int, *, lib=None):
    """Sec. 4.4 over a batch: q [B,H,nt,hd], k [B,H,n,hd], heads [B,nh]
    -> (kept [B,n2], v [B,n])."""
    lib = lib or load()
    Q, K = _f64(q), _f64(k)
    hs = _i32(heads)
    B, H, nt, hd = Q.shape
    n = K.shape[2]
    kept = np.empty((B, n2), np.int32)
    v = np.empty((B, n), np.float64)
    for b in range(B):
        rc = lib.orc_head_aware(_pd(Q[b]), _pd(K[b]), H, nt, n, hd, _pi(hs[b]), hs.shape[1],
                                int(n2), _pi(kept[b]), _pd(v[b]))
        if rc != 0:
            raise OracleError(f"orc_head_aware rc={rc}")
    return kept, v


def attention_in_model(q, k, lse, *, lib=None) -> np.ndarray:
    """One head, the visual slice of the model's softmax: q [nt, hd], k [n,
    hd], lse [nt] (log-sum-exp of the other keys' scaled logits) -> [nt, n]."""
    lib = lib or load()
    q, k, lse = _f64(q), _f64(k), _f64(lse)
    nt, hd = q.shape
    n = k.shape[0]
    A = np.empty((nt, n), np.float64)
    lib.orc_attention_in_model(_pd(q), _pd(k), _pd(lse), nt, n, hd, _pd(A))
    return A


def head_aware_in_model(q, k, heads, lse, n2: int, *, lib=None):
    """Sec. 4.4 on the in-model map over a batch: q [B,H,nt,hd], k
    [B,H,n,hd], heads [B,nh], lse [B,H,nt] -> (kept [B,n2], v [B,n])."""
    lib = lib or load()
    Q, K, L = _f64(q), _f64(k), _f64(lse)
    hs = _i32(heads)
    B, H, nt, hd = Q.shape
    n = K.shape[2]
    v = np.empty((B, n), np.float64)
    kept = np.empty((B, n2), np.int32)
    for b in range(B):
        rc = lib.orc_head_aware_score_in_model(_pd(Q[b]), _pd(K[b]), _pd(L[b]), H, nt, n, hd,
                                               _pi(hs[b]), hs.shape[1], _pd(v[b]))
        if rc != 0:
            raise OracleError(f"orc_head_aware_score_in_model rc={rc}")
        rc = lib.orc_topk(_pd(v[b]), n, int(n2), _pi(kept[b]))
        if rc != 0:
            raise OracleError(f"orc_topk rc={rc}")
    return kept, v


def head_confidence(q, k, *, lib=None) -> np.ndarray:
    """One sample: q [H, nt, hd], k [H, n, hd] -> C [H] (Sec. 4.4, equation
    for C^h)."""
    lib = lib or load()
    q, k = _f64(q), _f64(k)
    H, nt, hd = q.shape
    n = k.shape[1]
    c = np.empty(H, np.float64)
    rc = lib.orc_head_confidence(_pd(q), _pd(k), H, nt, n, hd, _pd(c))
    if rc != 0:
        raise OracleError(f"orc_head_confidence rc={rc}")
    return c


def visual_heads(q, k, n_vis: int, *, lib=None):
    """Sec. 4.4 over a batch: q [B,H,nt,hd], k [B,H,n,hd] -> (heads [B,n_vis]
    ascending, C [B,H])."""
    lib = lib or load()
    Q, K = _f64(q), _f64(k)
    B, H, nt, hd = Q.shape
    n = K.shape[2]
    heads = np.empty((B, n_vis), np.int32)
    conf = np.empty((B, H), np.float64)
    for b in range(B):
        rc = lib.orc_visual_heads(_pd(Q[b]), _pd(K[b]), H, nt, n, hd, int(n_vis), _pi(heads[b]),
                                  _pd(conf[b]))
        if rc != 0:
            raise OracleError(f"orc_visual_heads rc={rc}")
    return heads, conf


def head_confidence_in_model(q, k, lse, *, lib=None) -> np.ndarray:
    """One sample on the model's softmax domain: q [H, nt, hd], k [H, n, hd],
    lse [H, nt] (log-sum-exp of each row's scaled logits over the
    non-visual keys) -> C [H]."""
    lib = lib or load()
    q, k, lse = _f64(q), _f64(k), _f64(lse)
    H, nt, hd = q.shape
    n = k.shape[1]
    c = np.empty(H, np.float64)
    rc = lib.orc_head_confidence_in_model(_pd(q), _pd(k), _pd(lse), H, nt, n, hd, _pd(c))
    if rc != 0:
        raise OracleError(f"orc_head_confidence_in_model rc={rc}")
    return c


def visual_heads_in_model(q, k, lse, n_vis: int, *, lib=None):
    """Sec. 4.4 on the model's softmax domain over a batch: q [B,H,nt,hd],
    k [B,H,n,hd], lse [B,H,nt] -> (heads [B,n_vis] ascending, C [B,H])."""
    lib = lib or load()
    Q, K, L = _f64(q), _f64(k), _f64(lse)
    B, H, nt, hd = Q.shape
    n = K.shape[2]
    heads = np.empty((B, n_vis), np.int32)
    conf = np.empty((B, H), np.float64)
    for b in range(B):
        rc = lib.orc_visual_heads_in_model(_pd(Q[b]), _pd(K[b]), _pd(L[b]), H, nt, n, hd,
                                           int(n_vis), _pi(heads[b]), _pd(conf[b]))
        if rc != 0:
            raise OracleError(f"orc_visual_heads_in_model rc={rc}")
    return heads, conf


# ---------------------------------------------------------------- gather --

def gather(src: np.ndarray, idx, *, lib=None) -> np.ndarray:
    """Row compaction: src [B, G, n, ...] or [B, n, ...] (any dtype), idx
    [B, k] -> [B, G, k, ...] / [B, k, ...], copied byte for byte."""
    lib = lib or load()
    src = np.ascontiguousarray(src)
    ix = _i32(idx)
    B, k = ix.shape
    grouped = src.ndim >= 4
    if grouped:
        G, n = src.shape[1], src.shape[2]
        tail = src.shape[3:]
    else:
        G, n = 1, src.shape[1]
        tail = src.shape[2:]
    row_bytes = int(np.prod(tail, dtype=np.int64)) * src.itemsize
    out_shape = (B, G, k) + tuple(tail) if grouped else (B, k) + tuple(tail)
    dst = np.empty(out_shape, src.dtype)
    sb, sg, sr = n * G * row_bytes, n * row_bytes, row_bytes
    db, dg, dr = k * G * row_bytes, k * row_bytes, row_bytes
    rc = lib.orc_gather(src.ctypes.data_as(_U8), dst.ctypes.data_as(_U8), _pi(ix), B, n, k, G,
                        row_bytes, sb, sg, sr, db, dg, dr)
    if rc != 0:
        raise OracleError(f"orc_gather rc={rc}")
    return dst
