"""The C ABI without a GPU: the library loads, exports every entry point
declared in include/provip.h, and rejects bad arguments on the host before
anything is enqueued (these calls never reach a kernel launch)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "provip.h")


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(pv_[a-z_0-9]+)\s*\(", txt)))


@pytest.fixture(scope="module")
def lib():
    from paper_2608_25332_amd import provip
    return provip.load()


def test_header_declares_the_three_calls():
    names = _declared()
    for n in ("pv_prune_dedup", "pv_prune_head_aware", "pv_prune_gather",
              "pv_dedup_workspace_bytes", "pv_head_aware_workspace_bytes", "pv_status_string"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_exported_c_symbols_are_declared():
    """Every unmangled symbol the library exports is part of the header."""
    import shutil
    import subprocess
    from paper_2608_25332_amd import provip
    if shutil.which("nm") is None:
        pytest.skip("nm not available")
    out = subprocess.run(["nm", "-D", "--defined-only", provip.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    names = [l.split()[-1] for l in out.splitlines() if l.strip()]
    c_names = [n for n in names if not n.startswith("_Z") and not n.startswith("__")]
    assert set(c_names) <= set(_declared()), set(c_names) - set(_declared())


def test_status_strings(lib):
    for s in range(-9, 1):
        assert len(lib.pv_status_string(s)) > 0
    assert lib.pv_status_string(-99) == b"unknown status"
    assert lib.pv_version() >> 16 == 1


FAKE = 0x100000  # never dereferenced: every call below fails validation first


def _dedup(lib, vis=FAKE, anc=FAKE, B=1, Nv=64, Nt=16, d=256, dt=1, budget=32, kept=FAKE,
           ws=FAKE, wsb=1 << 40):
    return lib.pv_prune_dedup(vis, anc, B, Nv, Nt, d, dt, budget, kept, None, None, None, ws,
                              wsb, None)


def test_dedup_validation(lib):
    assert _dedup(lib, vis=None) == -1
    assert _dedup(lib, kept=None) == -1
    assert _dedup(lib, dt=7) == -5
    assert _dedup(lib, Nv=0) == -2
    assert _dedup(lib, d=100) == -2
    assert _dedup(lib, d=36) == -2
    assert _dedup(lib, d=4) == -2
    assert _dedup(lib, Nt=0) == -2
    assert _dedup(lib, Nv=20000) == -2
    assert _dedup(lib, budget=0) == -3
    assert _dedup(lib, budget=65) == -3
    assert _dedup(lib, ws=None) == -6
    assert _dedup(lib, wsb=16) == -6
    assert _dedup(lib, vis=FAKE + 4) == -8


def test_dedup_workspace_query(lib):
    a = lib.pv_dedup_workspace_bytes(1, 576, 64, 4096, 192, 1)
    b = lib.pv_dedup_workspace_bytes(16, 576, 64, 4096, 192, 1)
    assert 0 < a < b
    assert lib.pv_dedup_workspace_bytes(1, 576, 64, 4096, 0, 1) == 0
    assert lib.pv_dedup_workspace_bytes(1, 576, 64, 4096, 577, 1) == 0


def _heads(lib, heads, B=1, H=4, Nt=16, N=32, hd=64, dt=1, budget=8, q=FAKE, k=FAKE, kept=FAKE,
           ws=FAKE, wsb=1 << 40):
    hs = np.ascontiguousarray(np.asarray(heads, np.int32).reshape(B, -1))
    return lib.pv_prune_head_aware(q, k, hs.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                   hs.shape[1], B, H, Nt, N, hd, dt, budget, kept, None, ws, wsb,
                                   None)


def test_head_aware_validation(lib):
    assert _heads(lib, [1], q=None) == -1
    assert _heads(lib, [4]) == -4          # out of range
    assert _heads(lib, [-1]) == -4
    assert _heads(lib, [1, 1]) == -4       # repeated
    assert _heads(lib, [0, 1, 2, 3, 0]) == -4  # more heads than H
    assert _heads(lib, [1], hd=44) == -2
    assert _heads(lib, [1], hd=4) == -2
    assert _heads(lib, [1], hd=512) == -2
    assert _heads(lib, [1], N=0) == -2
    assert _heads(lib, [1], budget=0) == -3
    assert _heads(lib, [1], budget=33) == -3
    assert _heads(lib, [1], dt=3) == -5
    assert _heads(lib, [1], ws=None) == -6
    assert _heads(lib, [1], wsb=8) == -6
    assert _heads(lib, [1], q=FAKE + 8) == -8
    assert _heads(lib, [[0], [1], [4]], B=3) == -4   # a later sample is checked too


def test_head_aware_dev_validation(lib):
    f = lib.pv_prune_head_aware_dev

    def call(hd_ptr=FAKE, n_heads=2, H=4, hd=64, budget=8, q=FAKE, ws=FAKE, wsb=1 << 40):
        return f(q, FAKE, hd_ptr, n_heads, 1, H, 16, 32, hd, 1, budget, FAKE, None, ws, wsb, None)
    assert call(hd_ptr=None) == -1
    assert call(q=None) == -1
    assert call(n_heads=0) == -4
    assert call(n_heads=5) == -4           # more than H
    assert call(hd_ptr=FAKE + 2) == -8     # int32 list must be 4-byte aligned
    assert call(hd=44) == -2
    assert call(budget=33) == -3
    assert call(ws=None) == -6


def test_head_aware_ex_validation(lib):
    f = lib.pv_prune_head_aware_ex
    hs = np.zeros(2, np.int32)
    hp = hs.ctypes.data_as(ctypes.c_void_p)

    def call(hh=hp, hdev=None, lse=None, n_heads=2):
        return f(FAKE, FAKE, hh, hdev, n_heads, 1, 4, 16, 32, 64, 1, 8, lse, FAKE, None, FAKE,
                 1 << 40, None)
    assert call(hh=None) == -1            # no list at all
    assert call(hdev=FAKE) == -4          # two lists
    assert call(lse=FAKE + 2) == -8       # row_lse not 4-byte aligned
    hs[:] = [0, 0]
    assert call() == -4                   # the host list is still checked


def test_visual_heads_validation(lib):
    f = lib.pv_visual_heads
    assert lib.pv_visual_heads_workspace_bytes(1, 32, 64) > 0
    assert lib.pv_visual_heads_workspace_bytes(0, 32, 64) == 0

    def call(H=32, n_vis=6, Nt=64, N=192, hd=128, dt=1, out=FAKE, q=FAKE, ws=FAKE, wsb=1 << 40):
        return f(q, FAKE, 1, H, Nt, N, hd, dt, n_vis, out, None, ws, wsb, None)
    assert call(out=None) == -1
    assert call(q=None) == -1
    assert call(n_vis=0) == -4
    assert call(n_vis=33) == -4
    assert call(H=600, n_vis=6) == -4      # beyond PV_MAX_HEADS
    assert call(hd=44) == -2
    assert call(N=0) == -2
    assert call(dt=7) == -5
    assert call(ws=None) == -6
    assert call(wsb=4) == -6
    assert call(out=FAKE + 4) == -8


def test_critical_text_validation(lib):
    f = lib.pv_critical_text
    assert lib.pv_critical_text_workspace_bytes(1, 64, 4096, 1) > 0
    assert lib.pv_critical_text_workspace_bytes(1, 64, 4096, 9) == 0

    def call(text=FAKE, Nt=64, d=4096, dt=1, mask=FAKE, count=FAKE, ws=FAKE, wsb=1 << 40):
        return f(text, 1, Nt, d, dt, mask, count, None, ws, wsb, None)
    assert call(text=None) == -1
    assert call(mask=None) == -1
    assert call(count=None) == -1
    assert call(Nt=0) == -2
    assert call(Nt=1025) == -2
    assert call(d=100) == -2
    assert call(dt=2) == -5
    assert call(ws=None) == -6
    assert call(wsb=16) == -6
    assert call(mask=FAKE + 4) == -8


def test_masked_variants_validation(lib):
    d = lib.pv_prune_dedup_masked(FAKE, FAKE, None, 1, 576, 64, 4096, 1, 192, FAKE, None, None,
                                  None, FAKE, 1 << 40, None)
    assert d == -1
    d = lib.pv_prune_dedup_masked(FAKE, FAKE, FAKE + 2, 1, 576, 64, 4096, 1, 192, FAKE, None,
                                  None, None, FAKE, 1 << 40, None)
    assert d == -8
    d = lib.pv_prune_dedup_masked(FAKE, FAKE, FAKE, 1, 576, 64, 4096, 1, 577, FAKE, None, None,
                                  None, FAKE, 1 << 40, None)
    assert d == -3
    v = lib.pv_visual_heads_masked(FAKE, FAKE, None, 1, 32, 64, 192, 128, 1, 6, FAKE, None, FAKE,
                                   1 << 40, None)
    assert v == -1
    v = lib.pv_visual_heads_masked(FAKE, FAKE, FAKE + 1, 1, 32, 64, 192, 128, 1, 6, FAKE, None,
                                   FAKE, 1 << 40, None)
    assert v == -8


def test_gather_validation(lib):
    g = lib.pv_prune_gather
    args = dict(src=FAKE, dst=FAKE, idx=FAKE, B=1, n=8, k=4, G=1, rb=256)

    def call(**kw):
        a = {**args, **kw}
        return g(a["src"], a["dst"], a["idx"], a["B"], a["n"], a["k"], a["G"], a["rb"],
                 a["rb"] * a["n"], a["rb"] * a["n"], a["rb"], a["rb"] * a["k"], a["rb"] * a["k"],
                 a["rb"], None)
    assert call(src=None) == -1
    assert call(idx=None) == -1
    assert call(k=0) == -2
    assert call(rb=8) == -2
    assert call(rb=40) == -8
    assert call(dst=FAKE + 2) == -8


def test_gather_batch_validation(lib):
    from paper_2608_25332_amd import provip
    d = (provip.GatherDesc * 2)()
    for t in range(2):
        d[t].src, d[t].dst, d[t].n_src, d[t].groups, d[t].row_bytes = FAKE, FAKE, 8, 1, 256
        d[t].src_batch_stride = d[t].src_group_stride = 8 * 256
        d[t].src_row_stride = d[t].dst_row_stride = 256
        d[t].dst_batch_stride = d[t].dst_group_stride = 4 * 256
    g = lib.pv_prune_gather_batch
    assert g(None, 2, FAKE, 1, 4, None) == -1
    assert g(d, 0, FAKE, 1, 4, None) == -2
    assert g(d, 5, FAKE, 1, 4, None) == -2
    assert g(d, 2, FAKE, 1, 0, None) == -2
    assert g(d, 2, FAKE + 4, 1, 4, None) == -8
    d[1].row_bytes = 40
    assert g(d, 2, FAKE, 1, 4, None) == -8
    d[1].row_bytes = 256
    d[1].dst = None
    assert g(d, 2, FAKE, 1, 4, None) == -1


def test_select_topk_validation(lib):
    t = lib.pv_select_topk
    assert t(None, 1, 8, 4, FAKE, None, None, None) == -1
    assert t(FAKE, 1, 8, 4, None, None, None, None) == -1
    assert t(FAKE, 0, 8, 4, FAKE, None, None, None) == -2
    assert t(FAKE, 1, 0, 1, FAKE, None, None, None) == -2
    assert t(FAKE, 1, 16385, 4, FAKE, None, None, None) == -2
    assert t(FAKE, 1, 8, 0, FAKE, None, None, None) == -3
    assert t(FAKE, 1, 8, 9, FAKE, None, None, None) == -3
    assert t(FAKE + 4, 1, 8, 4, FAKE, None, None, None) == -8
    assert t(FAKE, 1, 8, 4, FAKE, FAKE + 8, None, None) == -8
    assert t(FAKE, 1, 8, 4, FAKE, None, FAKE + 12, None) == -8


def test_timed_reps_validation(lib):
    # reps < 1 is rejected before anything is enqueued
    rc = lib.pv_prune_dedup_timed(FAKE, FAKE, 1, 64, 16, 256, 1, 32, FAKE, None, None, None, FAKE,
                                  1 << 40, None, None, 0, 0, None, None)
    assert rc == -2
    hs = np.zeros((1, 1), np.int32)
    rc = lib.pv_prune_head_aware_timed(FAKE, FAKE, hs.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                       1, 1, 4, 16, 32, 64, 1, 8, FAKE, None, FAKE, 1 << 40, None,
                                       None, 0, 0, None, None)
    assert rc == -2


def test_timed_null_event_handle(lib):
    evs = (ctypes.c_void_p * 3)(FAKE, None, FAKE)
    rc = lib.pv_prune_dedup_timed(FAKE, FAKE, 1, 64, 16, 256, 1, 32, FAKE, None, None, None, FAKE,
                                  1 << 40, None, evs, 3, 1, None, None)
    assert rc == -1


def test_dedup_split_validation(lib):
    s = lib.pv_prune_dedup_split
    args = [FAKE, FAKE, 1, 64, 16, 256, 1, 32, FAKE, None, None, None, FAKE, 1 << 40, None]
    assert s(*args, None, FAKE, FAKE) == -1
    assert s(*args, FAKE, None, FAKE) == -1
    assert s(*args, FAKE, FAKE, None) == -1
    bad = list(args)
    bad[7] = 0  # budget
    assert s(*bad, FAKE, FAKE, FAKE) == -3


def test_every_kernel_launch_stub_is_defined():
    """A kernel whose host-side launch stub is missing leaves an undefined
    __device_stub__ symbol in the library; loading it would then fail on the
    GPU machine."""
    import shutil
    import subprocess
    from paper_2608_25332_amd import provip
    if shutil.which("nm") is None:
        pytest.skip("nm not available")
    out = subprocess.run(["nm", "-D", "--undefined-only", provip.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    missing = [l.split()[-1] for l in out.splitlines() if "__device_stub__" in l]
    assert not missing, missing[:5]


def _pipe(lib, heads=(1,), B=1, Nv=64, Nt=16, d=256, H=4, hd=64, dt=1, b1=32, b2=16, ws=FAKE,
          wsb=1 << 40, null_at=None, misalign_at=None):
    hs = np.ascontiguousarray(np.asarray(heads, dtype=np.int32).reshape(B, -1))
    ptrs = [FAKE] * 16  # vis anchors q k_full v_full, then the 11 outputs
    if null_at is not None:
        ptrs[null_at] = None
    if misalign_at is not None:
        ptrs[misalign_at] = FAKE + 8
    return lib.pv_prune_pipeline(*ptrs[:5], hs.ctypes.data_as(ctypes.c_void_p), hs.shape[1], B,
                                 Nv, Nt, d, H, hd, dt, b1, b2, *ptrs[5:], ws, wsb, None)


def test_pipeline_validation(lib):
    for i in range(16):
        assert _pipe(lib, null_at=i) == -1, i   # every pointer is required
    assert _pipe(lib, ws=None) == -6
    assert _pipe(lib, wsb=8) == -6
    assert _pipe(lib, b1=0) == -3
    assert _pipe(lib, b1=65) == -3
    assert _pipe(lib, b2=33) == -3              # budget2 counts the budget1 kept tokens
    assert _pipe(lib, heads=(4,)) == -4
    assert _pipe(lib, heads=(1, 1)) == -4
    assert _pipe(lib, d=100) == -2
    assert _pipe(lib, hd=44) == -2
    assert _pipe(lib, dt=3) == -5
    assert _pipe(lib, misalign_at=3) == -8
    assert _pipe(lib, misalign_at=12) == -8
    for f in (lib.pv_prune_pipeline, lib.pv_prune_pipeline_separate):
        hs = np.zeros((1, 1), np.int32)
        assert f(None, *[FAKE] * 4, hs.ctypes.data_as(ctypes.c_void_p), 1, 1, 64, 16, 256, 4, 64,
                 1, 32, 16, *[FAKE] * 11, FAKE, 1 << 40, None) == -1


def test_pipeline_workspace_query(lib):
    f = lib.pv_pipeline_workspace_bytes
    small = f(1, 576, 64, 4096, 32, 128, 4, 192, 64, 1)
    dedup = lib.pv_dedup_workspace_bytes(1, 576, 64, 4096, 192, 1)
    head = lib.pv_head_aware_workspace_bytes(1, 32, 64, 192, 128, 4, 64, 1)
    assert small >= dedup and small >= head
    assert f(16, 576, 64, 4096, 32, 128, 4, 192, 64, 1) > small
    assert f(1, 576, 64, 4096, 32, 128, 4, 0, 64, 1) == 0


def test_pipeline_timed_validation(lib):
    hs = np.ones((1, 1), np.int32)
    args = [FAKE] * 5 + [hs.ctypes.data_as(ctypes.c_void_p), 1, 1, 64, 16, 256, 4, 64, 1, 32, 16]
    args += [FAKE] * 11 + [FAKE, 1 << 40, None]
    evs = (ctypes.c_void_p * 3)(FAKE, None, FAKE)
    assert lib.pv_prune_pipeline_timed(*args, evs, 3, 0, None, None) == -2   # reps < 1
    assert lib.pv_prune_pipeline_timed(*args, evs, 3, 1, None, None) == -1   # a NULL event
    bad = list(args)
    bad[0] = None
    assert lib.pv_prune_pipeline_timed(*bad, None, 0, 1, None, None) == -1


def _noalloc(lib, heads=(1,), B=1, Nv=64, Nt=16, d=256, H=4, hd=64, dt=1, b1=32, b2=16,
             null_at=None):
    hs = np.ascontiguousarray(np.asarray(heads, dtype=np.int32).reshape(B, -1))
    ptrs = [FAKE] * 16
    if null_at is not None:
        ptrs[null_at] = None
    return lib.pv_prune_pipeline_noalloc(*ptrs[:5], hs.ctypes.data_as(ctypes.c_void_p),
                                         hs.shape[1], B, Nv, Nt, d, H, hd, dt, b1, b2, *ptrs[5:],
                                         None)


def test_pipeline_noalloc_rejects_on_the_host(lib):
    """The step on the static scratch: bad arguments and problems larger than
    the scratch are rejected before any device call (these return without a
    GPU)."""
    from paper_2608_25332_amd import provip
    assert _noalloc(lib, null_at=0) == -1
    assert _noalloc(lib, heads=(4,)) == -4
    assert _noalloc(lib, b1=65) == -3
    assert _noalloc(lib, d=100) == -2
    # the 13B 8-frame step fits; 16 samples of it do not
    big = dict(heads=[list(range(5))] * 16, B=16, Nv=4608, Nt=128, d=5120, H=40, hd=128,
               b1=1152, b2=512)
    assert lib.pv_pipeline_workspace_bytes(16, 4608, 128, 5120, 40, 128, 5, 1152, 512, 1) > \
        provip.PV_STATIC_SCRATCH_BYTES
    assert _noalloc(lib, **big) == -9
    assert lib.pv_pipeline_workspace_bytes(2, 4608, 128, 5120, 40, 128, 5, 1152, 512, 1) <= \
        provip.PV_STATIC_SCRATCH_BYTES
    assert b"scratch" in lib.pv_status_string(-9)


def _prog(lib, B=1, Nv=64, Nt=16, d=256, H=4, hd=64, dt=1, b1=32, nv=2, b2=16, b3=8, null_at=None,
          ws=FAKE, wsb=1 << 40):
    ptrs = [FAKE] * 18  # six inputs, then the twelve outputs
    if null_at is not None:
        ptrs[null_at] = None
    return lib.pv_prune_progressive(*ptrs[:6], B, Nv, Nt, d, H, hd, dt, b1, nv, b2, b3,
                                    *ptrs[6:], ws, wsb, None)


def test_progressive_validation(lib):
    """The progressive schedule's host checks (nothing is enqueued)."""
    assert _prog(lib, null_at=0) == -1          # text
    assert _prog(lib, null_at=6) == -1          # text_mask
    assert _prog(lib, null_at=17) == -1         # hidden3
    assert _prog(lib, b1=65) == -3
    assert _prog(lib, b2=33) == -3              # budget2 > budget1
    assert _prog(lib, b3=17) == -3              # budget3 > budget2
    assert _prog(lib, b3=0) == -3
    assert _prog(lib, nv=5) == -4               # more visual heads than heads
    assert _prog(lib, nv=0) == -4
    assert _prog(lib, hd=44) == -2
    assert _prog(lib, ws=None) == -6
    assert _prog(lib, wsb=64) == -6
    f = lib.pv_progressive_workspace_bytes
    assert f(1, 576, 64, 4096, 32, 128, 192, 6, 64, 32, 1) > 0
    assert f(1, 576, 64, 4096, 32, 128, 192, 6, 64, 65, 1) == 0


def test_ragged_widths_grow_the_workspace(lib):
    """Widths that are multiples of 8 but not of the streamed chunk (d = 4104,
    hd = 72 / 80 / 112) are accepted; their workspaces hold the zero-padded
    copies of the rows."""
    a = lib.pv_dedup_workspace_bytes(2, 576, 64, 4096, 192, 1)
    b = lib.pv_dedup_workspace_bytes(2, 576, 64, 4104, 192, 1)
    assert b >= a + 2 * (576 + 64) * 4160 * 2
    for hd in (72, 80, 112):
        w0 = lib.pv_head_aware_workspace_bytes(2, 8, 64, 300, 128, 4, 50, 1)
        w1 = lib.pv_head_aware_workspace_bytes(2, 8, 64, 300, hd, 4, 50, 1)
        assert w1 > 2 * 8 * (64 + 300) * ((hd + 31) // 32 * 32) * 2
        assert w0 < w1
        v1 = lib.pv_visual_heads_workspace_bytes_hd(2, 8, 64, 300, hd, 1)
        assert v1 > lib.pv_visual_heads_workspace_bytes(2, 8, 64)
    assert lib.pv_visual_heads_workspace_bytes_hd(2, 8, 64, 300, 128, 1) >= \
        lib.pv_visual_heads_workspace_bytes(2, 8, 64)
    assert lib.pv_critical_text_workspace_bytes(1, 64, 4104, 1) > \
        lib.pv_critical_text_workspace_bytes(1, 64, 4096, 1)
