"""ctypes binding of libprovip (the C ABI in include/provip.h).

Argument marshalling only: torch tensors supply device memory and the
current HIP stream; every step of the computation runs in the HIP kernels of
libprovip.so.  If the library is not built this module raises on first use;
there is no fallback path.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libprovip.so")

PV_OK = 0
PV_F32 = 0
PV_BF16 = 1

STATUS = {
    0: "PV_OK", -1: "PV_ERR_NULL", -2: "PV_ERR_SHAPE", -3: "PV_ERR_BUDGET", -4: "PV_ERR_HEADS",
    -5: "PV_ERR_DTYPE", -6: "PV_ERR_WORKSPACE", -7: "PV_ERR_HIP", -8: "PV_ERR_ALIGN",
    -9: "PV_ERR_SCRATCH",
}

# size of the library's static scratch array (pv_prune_pipeline_noalloc)
PV_STATIC_SCRATCH_BYTES = 64 << 20

_lib = None

_vp = ctypes.c_void_p
_i = ctypes.c_int
_i64 = ctypes.c_int64
_sz = ctypes.c_size_t


PV_MAX_GATHER = 4


class GatherDesc(ctypes.Structure):
    """pv_gather_desc of include/provip.h."""
    _fields_ = [("src", _vp), ("dst", _vp), ("n_src", _i), ("groups", _i), ("row_bytes", _i64),
                ("src_batch_stride", _i64), ("src_group_stride", _i64), ("src_row_stride", _i64),
                ("dst_batch_stride", _i64), ("dst_group_stride", _i64), ("dst_row_stride", _i64)]


class ProvipError(RuntimeError):
    def __init__(self, fn: str, status: int, lib=None):
        msg = lib.pv_status_string(status).decode() if lib is not None else ""
        super().__init__(f"{fn} failed: {STATUS.get(status, status)} ({msg})")
        self.status = status


def load(path: str = LIB_PATH):
    """Load libprovip.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libprovip.so is not built ({path}); run __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    lib.pv_status_string.argtypes = [_i]
    lib.pv_status_string.restype = ctypes.c_char_p
    lib.pv_version.argtypes = []
    lib.pv_version.restype = _i
    lib.pv_dedup_workspace_bytes.argtypes = [_i, _i, _i, _i, _i, _i]
    lib.pv_dedup_workspace_bytes.restype = _sz
    ded = [_vp, _vp, _i, _i, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.pv_prune_dedup.argtypes = ded
    lib.pv_prune_dedup.restype = _i
    names_t = ctypes.POINTER(ctypes.c_char_p)
    lib.pv_prune_dedup_timed.argtypes = ded + [ctypes.POINTER(_vp), _i, _i, ctypes.POINTER(_i),
                                              names_t]
    lib.pv_prune_dedup_timed.restype = _i
    lib.pv_prune_dedup_split.argtypes = ded + [_vp, _vp, _vp]
    lib.pv_prune_dedup_split.restype = _i
    lib.pv_head_aware_workspace_bytes.argtypes = [_i, _i, _i, _i, _i, _i, _i, _i]
    lib.pv_head_aware_workspace_bytes.restype = _sz
    ha = [_vp, _vp, ctypes.POINTER(ctypes.c_int32), _i, _i, _i, _i, _i, _i, _i, _i, _vp, _vp,
          _vp, _sz, _vp]
    lib.pv_prune_head_aware.argtypes = ha
    lib.pv_prune_head_aware.restype = _i
    lib.pv_prune_head_aware_timed.argtypes = ha + [ctypes.POINTER(_vp), _i, _i,
                                                   ctypes.POINTER(_i), names_t]
    lib.pv_prune_head_aware_timed.restype = _i
    timed_tail = [ctypes.POINTER(_vp), _i, _i, ctypes.POINTER(_i), names_t]
    dm = [_vp, _vp, _vp] + ded[2:]
    lib.pv_prune_dedup_masked.argtypes = dm
    lib.pv_prune_dedup_masked.restype = _i
    lib.pv_prune_dedup_masked_timed.argtypes = dm + timed_tail
    lib.pv_prune_dedup_masked_timed.restype = _i
    lib.pv_critical_text_workspace_bytes.argtypes = [_i, _i, _i, _i]
    lib.pv_critical_text_workspace_bytes.restype = _sz
    ct = [_vp, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.pv_critical_text.argtypes = ct
    lib.pv_critical_text.restype = _i
    lib.pv_critical_text_timed.argtypes = ct + timed_tail
    lib.pv_critical_text_timed.restype = _i
    had = [_vp, _vp, _vp] + ha[3:]
    lib.pv_prune_head_aware_dev.argtypes = had
    lib.pv_prune_head_aware_dev.restype = _i
    lib.pv_prune_head_aware_dev_timed.argtypes = had + [ctypes.POINTER(_vp), _i, _i,
                                                        ctypes.POINTER(_i), names_t]
    lib.pv_prune_head_aware_dev_timed.restype = _i
    hax = [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.pv_prune_head_aware_ex.argtypes = hax
    lib.pv_prune_head_aware_ex.restype = _i
    lib.pv_prune_head_aware_ex_timed.argtypes = hax + timed_tail
    lib.pv_prune_head_aware_ex_timed.restype = _i
    lib.pv_visual_heads_workspace_bytes.argtypes = [_i, _i, _i]
    lib.pv_visual_heads_workspace_bytes_hd.argtypes = [_i] * 6
    lib.pv_visual_heads_workspace_bytes_hd.restype = _sz
    lib.pv_visual_heads_workspace_bytes.restype = _sz
    vh = [_vp, _vp, _i, _i, _i, _i, _i, _i, _i, _vp, _vp, _vp, _sz, _vp]
    lib.pv_visual_heads.argtypes = vh
    lib.pv_visual_heads.restype = _i
    lib.pv_visual_heads_timed.argtypes = vh + [ctypes.POINTER(_vp), _i, _i, ctypes.POINTER(_i),
                                               names_t]
    lib.pv_visual_heads_timed.restype = _i
    vhm = [_vp, _vp, _vp] + vh[2:]
    lib.pv_visual_heads_masked.argtypes = vhm
    lib.pv_visual_heads_masked.restype = _i
    lib.pv_visual_heads_masked_timed.argtypes = vhm + timed_tail
    lib.pv_visual_heads_masked_timed.restype = _i
    vhx = [_vp, _vp, _vp, _vp] + vh[2:]
    lib.pv_visual_heads_ex.argtypes = vhx
    lib.pv_visual_heads_ex.restype = _i
    lib.pv_visual_heads_ex_timed.argtypes = vhx + timed_tail
    lib.pv_visual_heads_ex_timed.restype = _i
    lib.pv_prune_gather.argtypes = [_vp, _vp, _vp, _i, _i, _i, _i, _i64, _i64, _i64, _i64, _i64,
                                    _i64, _i64, _vp]
    lib.pv_prune_gather.restype = _i
    lib.pv_prune_gather_batch.argtypes = [ctypes.POINTER(GatherDesc), _i, _vp, _i, _i, _vp]
    lib.pv_prune_gather_batch.restype = _i
    lib.pv_select_topk.argtypes = [_vp, _i, _i, _i, _vp, _vp, _vp, _vp]
    lib.pv_select_topk.restype = _i
    lib.pv_pipeline_workspace_bytes.argtypes = [_i] * 10
    lib.pv_pipeline_workspace_bytes.restype = _sz
    pipe = [_vp] * 6 + [_i] * 10 + [_vp] * 12 + [_sz, _vp]
    lib.pv_prune_pipeline.argtypes = pipe
    lib.pv_prune_pipeline.restype = _i
    lib.pv_prune_pipeline_separate.argtypes = pipe
    lib.pv_prune_pipeline_separate.restype = _i
    lib.pv_prune_pipeline_timed.argtypes = pipe + timed_tail
    lib.pv_prune_pipeline_timed.restype = _i
    lib.pv_progressive_workspace_bytes.argtypes = [_i] * 11
    lib.pv_progressive_workspace_bytes.restype = _sz
    lib.pv_prune_progressive.argtypes = [_vp] * 6 + [_i] * 11 + [_vp] * 12 + [_vp, _sz, _vp]
    lib.pv_prune_progressive.restype = _i
    lib.pv_prune_pipeline_noalloc.argtypes = [_vp] * 6 + [_i] * 10 + [_vp] * 11 + [_vp]
    lib.pv_prune_pipeline_noalloc.restype = _i
    _lib = lib
    return lib


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return PV_BF16
    if t.dtype == torch.float32:
        return PV_F32
    raise TypeError(f"unsupported dtype {t.dtype}; use bfloat16 or float32")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _stream(device: torch.device):
    return torch.cuda.current_stream(device).cuda_stream


def _check(fn: str, rc: int, lib):
    if rc != PV_OK:
        raise ProvipError(fn, rc, lib)


def _contig(t: torch.Tensor, name: str) -> torch.Tensor:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _events_array(events: Optional[Sequence]):
    """(event handle array, count, kernel-name array) for the *_timed calls."""
    if not events:
        return None, 0, None
    arr = (_vp * len(events))(*[e.cuda_event if hasattr(e, "cuda_event") else e for e in events])
    return arr, len(events), (ctypes.c_char_p * len(events))()


def _names(names_arr, n: int):
    if names_arr is None:
        return []
    return [names_arr[i].decode() for i in range(n) if names_arr[i] is not None]


# ----------------------------------------------------------------------------
def pv_dedup_workspace_bytes(B: int, Nv: int, Nt: int, d: int, budget: int, dtype: int) -> int:
    return int(load().pv_dedup_workspace_bytes(B, Nv, Nt, d, budget, dtype))


def pv_prune_dedup(vis: torch.Tensor, anchors: torch.Tensor, budget: int, *,
                   want_score: bool = True, want_assign: bool = True, want_merged: bool = True,
                   out: Optional[dict] = None, workspace: Optional[torch.Tensor] = None,
                   events: Optional[Sequence] = None, reps: int = 1, split=None,
                   anchor_mask: Optional[torch.Tensor] = None):
    """Pruning before the LLM.  vis [B, Nv, d], anchors [B, Nt, d] (same dtype).
    Returns dict(kept [B,budget] int32, score [B,Nv] f32 | None,
    assign [B,Nv] int32 | None, merged [B,budget,d] | None, n_kernels).
    events / reps: see pv_prune_dedup_timed (profiling only).
    anchor_mask: int32 [B, Nt] on the device (e.g. pv_critical_text's mask):
    only the rows set are anchors (pv_prune_dedup_masked).
    split = (merge_stream, selected, merged_done) (a torch stream and two torch
    events, already recorded once so that their HIP events exist): runs
    pv_prune_dedup_split; assign and merged are ready after merged_done."""
    lib = load()
    _contig(vis, "vis")
    _contig(anchors, "anchors")
    B, Nv, d = vis.shape
    Bt, Nt, dt_ = anchors.shape
    if Bt != B or dt_ != d or anchors.dtype != vis.dtype:
        raise ValueError("anchors must be [B, Nt, d] with the dtype of vis")
    code = _dtype_code(vis)
    dev = vis.device
    o = out if out is not None else {}
    kept = o.get("kept")
    if kept is None:
        kept = torch.empty((B, budget), dtype=torch.int32, device=dev)
    score = o.get("score") if want_score else None
    if want_score and score is None:
        score = torch.empty((B, Nv), dtype=torch.float32, device=dev)
    assign = o.get("assign") if want_assign else None
    if want_assign and assign is None:
        assign = torch.empty((B, Nv), dtype=torch.int32, device=dev)
    merged = o.get("merged") if want_merged else None
    if want_merged and merged is None:
        merged = torch.empty((B, budget, d), dtype=vis.dtype, device=dev)
    nbytes = lib.pv_dedup_workspace_bytes(B, Nv, Nt, d, budget, code)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    if split is not None:
        if events:
            raise ValueError("events and split cannot be combined")
        if anchor_mask is not None:
            raise ValueError("anchor_mask and split cannot be combined")
        merge_stream, selected, merged_done = split
        rc = lib.pv_prune_dedup_split(vis.data_ptr(), anchors.data_ptr(), B, Nv, Nt, d, code,
                                      int(budget), kept.data_ptr(), _ptr(score), _ptr(assign),
                                      _ptr(merged), workspace.data_ptr(), workspace.numel(),
                                      _stream(dev), merge_stream.cuda_stream,
                                      selected.cuda_event, merged_done.cuda_event)
        _check("pv_prune_dedup_split", rc, lib)
        # the merge stream reads vis, kept and the workspace and writes assign
        # and merged after this call returns: keep the caching allocator from
        # handing any of them to another allocation until that work is done
        for t in (vis, anchors, kept, score, assign, merged, workspace):
            if t is not None:
                t.record_stream(merge_stream)
        return {"kept": kept, "score": score, "assign": assign, "merged": merged,
                "n_kernels": None, "kernel_names": [], "workspace": workspace}
    ev, nev, nm = _events_array(events)
    nk = _i(0)
    if anchor_mask is not None:
        if split is not None:
            raise ValueError("anchor_mask and split cannot be combined")
        _check_mask(anchor_mask, B, Nt, dev, "anchor_mask")
        rc = lib.pv_prune_dedup_masked_timed(vis.data_ptr(), anchors.data_ptr(),
                                             anchor_mask.data_ptr(), B, Nv, Nt, d, code,
                                             int(budget), kept.data_ptr(), _ptr(score),
                                             _ptr(assign), _ptr(merged), workspace.data_ptr(),
                                             workspace.numel(), _stream(dev), ev, nev, int(reps),
                                             ctypes.byref(nk), nm)
    else:
        rc = lib.pv_prune_dedup_timed(vis.data_ptr(), anchors.data_ptr(), B, Nv, Nt, d, code,
                                      int(budget), kept.data_ptr(), _ptr(score), _ptr(assign),
                                      _ptr(merged), workspace.data_ptr(), workspace.numel(),
                                      _stream(dev), ev, nev, int(reps), ctypes.byref(nk), nm)
    _check("pv_prune_dedup", rc, lib)
    return {"kept": kept, "score": score, "assign": assign, "merged": merged,
            "n_kernels": nk.value, "kernel_names": _names(nm, min(nk.value, max(nev - 1, 0))),
            "workspace": workspace}


def pv_head_aware_workspace_bytes(B: int, H: int, Nt: int, N: int, hd: int, n_heads: int,
                                  budget: int, dtype: int) -> int:
    return int(load().pv_head_aware_workspace_bytes(B, H, Nt, N, hd, n_heads, budget, dtype))


def _check_mask(m: torch.Tensor, B: int, Nt: int, dev, name: str):
    if (m.dtype != torch.int32 or tuple(m.shape) != (B, Nt) or m.device != dev
            or not m.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous int32 [B, Nt] tensor on {dev}")


def pv_critical_text_workspace_bytes(B: int, Nt: int, d: int, dtype: int) -> int:
    return int(load().pv_critical_text_workspace_bytes(B, Nt, d, dtype))


def pv_critical_text(text: torch.Tensor, *, want_r: bool = True, out: Optional[dict] = None,
                     workspace: Optional[torch.Tensor] = None,
                     events: Optional[Sequence] = None, reps: int = 1):
    """Critical text tokens.  text [B, Nt, d].  Returns dict(mask [B,Nt]
    int32 (1 = critical), count [B] int32, r [B,Nt] f32 | None)."""
    lib = load()
    _contig(text, "text")
    B, Nt, d = text.shape
    code = _dtype_code(text)
    dev = text.device
    o = out if out is not None else {}
    mask = o.get("mask")
    if mask is None:
        mask = torch.empty((B, Nt), dtype=torch.int32, device=dev)
    count = o.get("count")
    if count is None:
        count = torch.empty((B,), dtype=torch.int32, device=dev)
    r = o.get("r") if want_r else None
    if want_r and r is None:
        r = torch.empty((B, Nt), dtype=torch.float32, device=dev)
    nbytes = lib.pv_critical_text_workspace_bytes(B, Nt, d, code)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    ev, nev, nm = _events_array(events)
    nk = _i(0)
    rc = lib.pv_critical_text_timed(text.data_ptr(), B, Nt, d, code, mask.data_ptr(),
                                    count.data_ptr(), _ptr(r), workspace.data_ptr(),
                                    workspace.numel(), _stream(dev), ev, nev, int(reps),
                                    ctypes.byref(nk), nm)
    _check("pv_critical_text", rc, lib)
    return {"mask": mask, "count": count, "r": r, "n_kernels": nk.value,
            "kernel_names": _names(nm, min(nk.value, max(nev - 1, 0))), "workspace": workspace}


def pv_visual_heads_workspace_bytes(B: int, H: int, Nt: int) -> int:
    return int(load().pv_visual_heads_workspace_bytes(B, H, Nt))


def pv_prune_head_aware(q: torch.Tensor, k: torch.Tensor, heads, budget: int, *,
                        want_score: bool = True, out: Optional[dict] = None,
                        workspace: Optional[torch.Tensor] = None,
                        events: Optional[Sequence] = None, reps: int = 1,
                        row_lse: Optional[torch.Tensor] = None):
    """Head-aware pruning.  q [B,H,Nt,hd], k [B,H,N,hd] (same dtype), heads:
    host int sequence [B, n_heads], or an int32 tensor [B, n_heads] on q's
    device (pv_prune_head_aware_dev: e.g. the list pv_visual_heads wrote).
    row_lse: float32 [B,H,Nt] on the device, the log-sum-exp of each row's
    scaled logits over the non-visual keys (pv_prune_head_aware_ex).
    Returns dict(kept [B,budget] int32, score [B,N] f32 | None, n_kernels).
    events / reps: see pv_prune_head_aware_timed (profiling only)."""
    import numpy as np

    lib = load()
    _contig(q, "q")
    _contig(k, "k")
    B, H, Nt, hd = q.shape
    Bk, Hk, N, hdk = k.shape
    if (Bk, Hk, hdk) != (B, H, hd) or k.dtype != q.dtype:
        raise ValueError("k must be [B, H, N, hd] with the dtype of q")
    on_dev = isinstance(heads, torch.Tensor) and heads.device.type != "cpu"
    if on_dev:
        if heads.dtype != torch.int32 or heads.dim() != 2 or heads.shape[0] != B:
            raise ValueError("a device head list must be int32 [B, n_heads]")
        _contig(heads, "heads")
        hs = heads
    else:
        hs = np.ascontiguousarray(np.asarray(heads, dtype=np.int32).reshape(B, -1))
    n_heads = hs.shape[1]
    code = _dtype_code(q)
    dev = q.device
    o = out if out is not None else {}
    kept = o.get("kept")
    if kept is None:
        kept = torch.empty((B, budget), dtype=torch.int32, device=dev)
    score = o.get("score") if want_score else None
    if want_score and score is None:
        score = torch.empty((B, N), dtype=torch.float32, device=dev)
    nbytes = lib.pv_head_aware_workspace_bytes(B, H, Nt, N, hd, n_heads, budget, code)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    ev, nev, nm = _events_array(events)
    nk = _i(0)
    if row_lse is not None:
        if (row_lse.dtype != torch.float32 or tuple(row_lse.shape) != (B, H, Nt)
                or row_lse.device != dev or not row_lse.is_contiguous()):
            raise ValueError(f"row_lse must be a contiguous float32 [B, H, Nt] tensor on {dev}")
        hh = None if on_dev else hs.ctypes.data_as(ctypes.c_void_p)
        hd_ptr = hs.data_ptr() if on_dev else None
        rc = lib.pv_prune_head_aware_ex_timed(q.data_ptr(), k.data_ptr(), hh, hd_ptr, n_heads, B,
                                              H, Nt, N, hd, code, int(budget), row_lse.data_ptr(),
                                              kept.data_ptr(), _ptr(score), workspace.data_ptr(),
                                              workspace.numel(), _stream(dev), ev, nev, int(reps),
                                              ctypes.byref(nk), nm)
    elif on_dev:
        rc = lib.pv_prune_head_aware_dev_timed(q.data_ptr(), k.data_ptr(), hs.data_ptr(), n_heads,
                                               B, H, Nt, N, hd, code, int(budget), kept.data_ptr(),
                                               _ptr(score), workspace.data_ptr(), workspace.numel(),
                                               _stream(dev), ev, nev, int(reps), ctypes.byref(nk),
                                               nm)
    else:
        rc = lib.pv_prune_head_aware_timed(q.data_ptr(), k.data_ptr(),
                                           hs.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                           n_heads, B, H, Nt, N, hd, code, int(budget),
                                           kept.data_ptr(), _ptr(score), workspace.data_ptr(),
                                           workspace.numel(), _stream(dev), ev, nev, int(reps),
                                           ctypes.byref(nk), nm)
    _check("pv_prune_head_aware", rc, lib)
    return {"kept": kept, "score": score, "n_kernels": nk.value,
            "kernel_names": _names(nm, min(nk.value, max(nev - 1, 0))), "workspace": workspace}


def pv_visual_heads(q: torch.Tensor, k: torch.Tensor, n_vis: int, *, want_conf: bool = True,
                    out: Optional[dict] = None, workspace: Optional[torch.Tensor] = None,
                    events: Optional[Sequence] = None, reps: int = 1,
                    row_mask: Optional[torch.Tensor] = None,
                    row_lse: Optional[torch.Tensor] = None):
    """Visual-head identification.  q [B,H,Nt,hd], k [B,H,N,hd].  Returns
    dict(heads [B,n_vis] int32 on the device, ascending; conf [B,H] f32 |
    None, n_kernels).  The head list can go straight to pv_prune_head_aware.
    row_mask: int32 [B, Nt] on the device: the confidence sums over the rows
    set only (pv_visual_heads_masked).  row_lse: float32 [B, H, Nt] on the
    device: the log-sum-exp of each row's scaled logits over the non-visual
    keys, so that the variance is taken on the model's softmax domain
    (pv_visual_heads_ex)."""
    lib = load()
    _contig(q, "q")
    _contig(k, "k")
    B, H, Nt, hd = q.shape
    Bk, Hk, N, hdk = k.shape
    if (Bk, Hk, hdk) != (B, H, hd) or k.dtype != q.dtype:
        raise ValueError("k must be [B, H, N, hd] with the dtype of q")
    dev = q.device
    o = out if out is not None else {}
    heads = o.get("heads")
    if heads is None:
        heads = torch.empty((B, n_vis), dtype=torch.int32, device=dev)
    conf = o.get("conf") if want_conf else None
    if want_conf and conf is None:
        conf = torch.empty((B, H), dtype=torch.float32, device=dev)
    nbytes = lib.pv_visual_heads_workspace_bytes_hd(B, H, Nt, N, hd, _dtype_code(q))
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    ev, nev, nm = _events_array(events)
    nk = _i(0)
    if row_lse is not None:
        if row_mask is not None:
            _check_mask(row_mask, B, Nt, dev, "row_mask")
        if (tuple(row_lse.shape) != (B, H, Nt) or row_lse.dtype != torch.float32
                or row_lse.device != dev or not row_lse.is_contiguous()):
            raise ValueError("row_lse must be a contiguous float32 [B, H, Nt] device tensor")
        rc = lib.pv_visual_heads_ex_timed(q.data_ptr(), k.data_ptr(), _ptr(row_mask),
                                          row_lse.data_ptr(), B, H, Nt, N, hd, _dtype_code(q),
                                          int(n_vis), heads.data_ptr(), _ptr(conf),
                                          workspace.data_ptr(), workspace.numel(), _stream(dev),
                                          ev, nev, int(reps), ctypes.byref(nk), nm)
    elif row_mask is not None:
        _check_mask(row_mask, B, Nt, dev, "row_mask")
        rc = lib.pv_visual_heads_masked_timed(q.data_ptr(), k.data_ptr(), row_mask.data_ptr(), B,
                                              H, Nt, N, hd, _dtype_code(q), int(n_vis),
                                              heads.data_ptr(), _ptr(conf), workspace.data_ptr(),
                                              workspace.numel(), _stream(dev), ev, nev, int(reps),
                                              ctypes.byref(nk), nm)
    else:
        rc = lib.pv_visual_heads_timed(q.data_ptr(), k.data_ptr(), B, H, Nt, N, hd,
                                       _dtype_code(q), int(n_vis), heads.data_ptr(), _ptr(conf),
                                       workspace.data_ptr(), workspace.numel(), _stream(dev), ev,
                                       nev, int(reps), ctypes.byref(nk), nm)
    _check("pv_visual_heads", rc, lib)
    return {"heads": heads, "conf": conf, "n_kernels": nk.value,
            "kernel_names": _names(nm, min(nk.value, max(nev - 1, 0))), "workspace": workspace}


def _gather_geometry(src: torch.Tensor, B: int, k: int):
    """(groups, n_src, row_bytes, out_shape) of a contiguous [B, N, ...] or
    [B, G, N, hd] tensor (4-D tensors are K/V caches with G head groups)."""
    if src.dim() == 4:
        _, G, n, hd = src.shape
        return G, n, hd * src.element_size(), (B, G, k, hd)
    G, n = 1, src.shape[1]
    per_row = 1
    for x in src.shape[2:]:
        per_row *= int(x)
    return G, n, per_row * src.element_size(), (B, k) + tuple(src.shape[2:])


def pv_prune_gather(src: torch.Tensor, idx: torch.Tensor, *, out: Optional[torch.Tensor] = None):
    """Order-preserving compaction of rows.  src [B, N, ...] (groups = 1) or
    [B, G, N, hd] (K/V caches, G head groups); idx [B, k] int32 device.
    Returns dst [B, k, ...] / [B, G, k, hd]."""
    lib = load()
    _contig(src, "src")
    _contig(idx, "idx")
    if idx.dtype != torch.int32:
        raise TypeError("idx must be int32")
    B, k = idx.shape
    G, n, row_bytes, shape = _gather_geometry(src, B, k)
    if out is None:
        out = torch.empty(shape, dtype=src.dtype, device=src.device)
    sb, sg, sr = n * G * row_bytes, n * row_bytes, row_bytes
    db, dg, dr = k * G * row_bytes, k * row_bytes, row_bytes
    rc = lib.pv_prune_gather(src.data_ptr(), out.data_ptr(), idx.data_ptr(), B, n, k, G,
                             row_bytes, sb, sg, sr, db, dg, dr, _stream(src.device))
    _check("pv_prune_gather", rc, lib)
    return out


def pv_select_topk(scores: torch.Tensor, k: int, *, want_rest: bool = False,
                   want_slot: bool = False, out: Optional[dict] = None):
    """Top-k of float32 scores [B, n] (or [n]); ties go to the lower index.
    Returns dict(kept [B,k] int32 ascending, rest [B,n-k] | None,
    slot_of [B,n] | None), shaped like the input's batch."""
    lib = load()
    _contig(scores, "scores")
    if scores.dtype != torch.float32:
        raise TypeError("scores must be float32")
    flat = scores.dim() == 1
    s2 = scores.view(1, -1) if flat else scores
    B, n = s2.shape
    dev = scores.device
    o = out if out is not None else {}

    def buf(name, want, shape):
        if not want:
            return None
        t = o.get(name)
        return t if t is not None else torch.empty(shape, dtype=torch.int32, device=dev)

    kept = buf("kept", True, (B, k))
    rest = buf("rest", want_rest, (B, n - k))
    slot = buf("slot_of", want_slot, (B, n))
    rc = lib.pv_select_topk(s2.data_ptr(), B, n, int(k), kept.data_ptr(), _ptr(rest), _ptr(slot),
                            _stream(dev))
    _check("pv_select_topk", rc, lib)
    res = {"kept": kept, "rest": rest, "slot_of": slot}
    if flat:
        res = {key: (v.view(-1) if v is not None else None) for key, v in res.items()}
    return res


def pv_prune_gather_batch(srcs: Sequence[torch.Tensor], idx: torch.Tensor, *,
                          outs: Optional[Sequence[torch.Tensor]] = None):
    """pv_prune_gather of up to PV_MAX_GATHER tensors sharing idx, in one launch."""
    lib = load()
    _contig(idx, "idx")
    if idx.dtype != torch.int32:
        raise TypeError("idx must be int32")
    B, k = idx.shape
    if not 1 <= len(srcs) <= PV_MAX_GATHER:
        raise ValueError(f"1..{PV_MAX_GATHER} tensors per batch")
    descs = (GatherDesc * len(srcs))()
    res = []
    for t, src in enumerate(srcs):
        _contig(src, "src")
        G, n, row_bytes, shape = _gather_geometry(src, B, k)
        out = outs[t] if outs is not None else torch.empty(shape, dtype=src.dtype, device=src.device)
        d = descs[t]
        d.src, d.dst, d.n_src, d.groups, d.row_bytes = src.data_ptr(), out.data_ptr(), n, G, row_bytes
        d.src_batch_stride, d.src_group_stride, d.src_row_stride = n * G * row_bytes, n * row_bytes, row_bytes
        d.dst_batch_stride, d.dst_group_stride, d.dst_row_stride = k * G * row_bytes, k * row_bytes, row_bytes
        res.append(out)
    rc = lib.pv_prune_gather_batch(descs, len(srcs), idx.data_ptr(), B, k, _stream(idx.device))
    _check("pv_prune_gather_batch", rc, lib)
    return res


# ----------------------------------------------------------------------------
PIPELINE_OUTPUTS = ("kept1", "score1", "assign", "merged", "k1", "v1", "kept2", "score2",
                    "hidden2", "k2", "v2")


def pv_pipeline_workspace_bytes(B: int, Nv: int, Nt: int, d: int, H: int, hd: int, n_heads: int,
                                budget1: int, budget2: int, dtype: int) -> int:
    return int(load().pv_pipeline_workspace_bytes(B, Nv, Nt, d, H, hd, n_heads, budget1, budget2,
                                                  dtype))


def pv_prune_pipeline(vis: torch.Tensor, anchors: torch.Tensor, q: torch.Tensor,
                      k_full: torch.Tensor, v_full: torch.Tensor, heads, budget1: int,
                      budget2: int, *, out: Optional[dict] = None,
                      workspace: Optional[torch.Tensor] = None, separate: bool = False,
                      events: Optional[Sequence] = None, reps: int = 1):
    """The whole pruning step (pv_prune_pipeline): dedup with the merge, the
    K/V rows of the budget1 kept tokens, head-aware score and top-budget2,
    and the compaction of the merged hidden rows, K and V.
    vis [B,Nv,d], anchors [B,Nt,d], q [B,H,Nt,hd], k_full / v_full
    [B,H,Nv,hd] (one dtype), heads: host ints [B, n_heads].  Returns a dict
    with PIPELINE_OUTPUTS (see include/provip.h for their shapes).
    separate=True runs every kernel in its own launch
    (pv_prune_pipeline_separate).  events / reps: see pv_prune_pipeline_timed
    (profiling only); the result then also holds n_kernels and
    kernel_names."""
    import numpy as np

    lib = load()
    for t, n in ((vis, "vis"), (anchors, "anchors"), (q, "q"), (k_full, "k_full"),
                 (v_full, "v_full")):
        _contig(t, n)
    B, Nv, d = vis.shape
    _, H, Nt, hd = q.shape
    if (tuple(anchors.shape) != (B, Nt, d) or tuple(k_full.shape) != (B, H, Nv, hd)
            or tuple(v_full.shape) != (B, H, Nv, hd)
            or len({t.dtype for t in (vis, anchors, q, k_full, v_full)}) != 1):
        raise ValueError("anchors [B,Nt,d], q [B,H,Nt,hd], k_full/v_full [B,H,Nv,hd], one dtype")
    hs = np.ascontiguousarray(np.asarray(heads, dtype=np.int32).reshape(B, -1))
    n_heads = hs.shape[1]
    code = _dtype_code(vis)
    dev, dt = vis.device, vis.dtype
    i32, f32 = torch.int32, torch.float32
    shapes = {"kept1": ((B, budget1), i32), "score1": ((B, Nv), f32), "assign": ((B, Nv), i32),
              "merged": ((B, budget1, d), dt), "k1": ((B, H, budget1, hd), dt),
              "v1": ((B, H, budget1, hd), dt), "kept2": ((B, budget2), i32),
              "score2": ((B, budget1), f32), "hidden2": ((B, budget2, d), dt),
              "k2": ((B, H, budget2, hd), dt), "v2": ((B, H, budget2, hd), dt)}
    o = dict(out) if out is not None else {}
    for name in PIPELINE_OUTPUTS:
        if o.get(name) is None:
            shp, ty = shapes[name]
            o[name] = torch.empty(shp, dtype=ty, device=dev)
        else:
            _contig(o[name], name)
    nbytes = lib.pv_pipeline_workspace_bytes(B, Nv, Nt, d, H, hd, n_heads, budget1, budget2, code)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    args = [vis.data_ptr(), anchors.data_ptr(), q.data_ptr(), k_full.data_ptr(),
            v_full.data_ptr(), hs.ctypes.data_as(ctypes.c_void_p), n_heads, B, Nv, Nt, d, H, hd,
            code, budget1, budget2, *[o[n].data_ptr() for n in PIPELINE_OUTPUTS],
            workspace.data_ptr(), workspace.numel(), _stream(dev)]
    if events is not None:
        if separate:
            raise ValueError("events are for the shared-launch step")
        ev, nev, nm = _events_array(events)
        nk = _i(0)
        rc = lib.pv_prune_pipeline_timed(*args, ev, nev, reps, ctypes.byref(nk), nm)
        _check("pv_prune_pipeline_timed", rc, lib)
        o["n_kernels"] = nk.value
        o["kernel_names"] = _names(nm, nk.value)
    else:
        fn = lib.pv_prune_pipeline_separate if separate else lib.pv_prune_pipeline
        rc = fn(*args)
        _check("pv_prune_pipeline_separate" if separate else "pv_prune_pipeline", rc, lib)
    o["workspace"] = workspace
    return o


def pv_prune_pipeline_noalloc(vis: torch.Tensor, anchors: torch.Tensor, q: torch.Tensor,
                              k_full: torch.Tensor, v_full: torch.Tensor, heads, budget1: int,
                              budget2: int, *, out: dict):
    """The whole step with the library's static scratch instead of a
    workspace (pv_prune_pipeline_noalloc): nothing is allocated on the
    device, so every output must be passed in `out` (PIPELINE_OUTPUTS, the
    shapes of pv_prune_pipeline's).  Calls that overlap in time on one GPU
    race on the scratch."""
    import numpy as np

    lib = load()
    for t, n in ((vis, "vis"), (anchors, "anchors"), (q, "q"), (k_full, "k_full"),
                 (v_full, "v_full")):
        _contig(t, n)
    B, Nv, d = vis.shape
    _, H, Nt, hd = q.shape
    hs = np.ascontiguousarray(np.asarray(heads, dtype=np.int32).reshape(B, -1))
    missing = [n for n in PIPELINE_OUTPUTS if out.get(n) is None]
    if missing:
        raise ValueError(f"pv_prune_pipeline_noalloc allocates nothing: pass {missing} in out")
    for n in PIPELINE_OUTPUTS:
        _contig(out[n], n)
    rc = lib.pv_prune_pipeline_noalloc(
        vis.data_ptr(), anchors.data_ptr(), q.data_ptr(), k_full.data_ptr(), v_full.data_ptr(),
        hs.ctypes.data_as(ctypes.c_void_p), hs.shape[1], B, Nv, Nt, d, H, hd, _dtype_code(vis),
        budget1, budget2, *[out[n].data_ptr() for n in PIPELINE_OUTPUTS], _stream(vis.device))
    _check("pv_prune_pipeline_noalloc", rc, lib)
    return out


PROGRESSIVE_OUTPUTS = ("text_mask", "kept1", "assign", "merged", "vis_heads", "conf", "kept2",
                       "score2", "hidden2", "kept3", "score3", "hidden3")


def pv_prune_progressive(text: torch.Tensor, vis: torch.Tensor, q_s: torch.Tensor,
                         k_s_all: torch.Tensor, q_m: torch.Tensor, k_m_all: torch.Tensor,
                         budget1: int, n_vis: int, budget2: int, budget3: int, *,
                         out: Optional[dict] = None, workspace: Optional[torch.Tensor] = None):
    """The progressive schedule in one call (pv_prune_progressive): critical
    text, pruning before the LLM on the critical rows, visual heads and
    head-aware pruning at the shallow layer (q_s, k_s_all), all-head pruning
    at the middle layer (q_m, k_m_all).  text [B,Nt,d], vis [B,Nv,d], q_*
    [B,H,Nt,hd], k_*_all [B,H,Nv,hd] (one dtype).  Returns a dict with
    PROGRESSIVE_OUTPUTS (shapes in include/provip.h)."""
    lib = load()
    for t, n in ((text, "text"), (vis, "vis"), (q_s, "q_s"), (k_s_all, "k_s_all"), (q_m, "q_m"),
                 (k_m_all, "k_m_all")):
        _contig(t, n)
    B, Nv, d = vis.shape
    _, H, Nt, hd = q_s.shape
    if (tuple(text.shape) != (B, Nt, d) or tuple(k_s_all.shape) != (B, H, Nv, hd)
            or tuple(q_m.shape) != (B, H, Nt, hd) or tuple(k_m_all.shape) != (B, H, Nv, hd)
            or len({t.dtype for t in (text, vis, q_s, k_s_all, q_m, k_m_all)}) != 1):
        raise ValueError("text [B,Nt,d], q_* [B,H,Nt,hd], k_*_all [B,H,Nv,hd], one dtype")
    code = _dtype_code(vis)
    dev, dt = vis.device, vis.dtype
    i32, f32 = torch.int32, torch.float32
    shapes = {"text_mask": ((B, Nt), i32), "kept1": ((B, budget1), i32),
              "assign": ((B, Nv), i32), "merged": ((B, budget1, d), dt),
              "vis_heads": ((B, n_vis), i32), "conf": ((B, H), f32),
              "kept2": ((B, budget2), i32), "score2": ((B, budget1), f32),
              "hidden2": ((B, budget2, d), dt), "kept3": ((B, budget3), i32),
              "score3": ((B, budget2), f32), "hidden3": ((B, budget3, d), dt)}
    o = dict(out) if out is not None else {}
    for name in PROGRESSIVE_OUTPUTS:
        if o.get(name) is None:
            shp, ty = shapes[name]
            o[name] = torch.empty(shp, dtype=ty, device=dev)
        else:
            _contig(o[name], name)
    nbytes = lib.pv_progressive_workspace_bytes(B, Nv, Nt, d, H, hd, budget1, n_vis, budget2,
                                                budget3, code)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    rc = lib.pv_prune_progressive(
        text.data_ptr(), vis.data_ptr(), q_s.data_ptr(), k_s_all.data_ptr(), q_m.data_ptr(),
        k_m_all.data_ptr(), B, Nv, Nt, d, H, hd, code, budget1, n_vis, budget2, budget3,
        *[o[n].data_ptr() for n in PROGRESSIVE_OUTPUTS], workspace.data_ptr(),
        workspace.numel(), _stream(dev))
    _check("pv_prune_progressive", rc, lib)
    o["workspace"] = workspace
    return o
