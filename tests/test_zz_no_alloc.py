"""pv_prune_pipeline_noalloc: the whole step on the library's static scratch
(no workspace, nothing allocated) against pv_prune_pipeline with a caller
workspace.  Both run the same kernels, so every output must match bit for
bit.  Three calls in a row on one GPU, each smaller than the one before
(the scratch keeps the previous call's contents)."""

from __future__ import annotations

import sys

import numpy as np
import pytest

from paper_2608_25332_amd import workloads as W
from parity_util import to_dev

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


def _inputs(w):
    dt = w.dtype
    return (to_dev(w.vis, dt), to_dev(w.anchors, dt), to_dev(w.q, dt), to_dev(w.k_full, dt),
            to_dev(w.v_full, dt))


def _assert_same(a, b, what):
    from paper_2608_25332_amd import provip
    for n in provip.PIPELINE_OUTPUTS:
        x = a[n].view(torch.uint8) if a[n].dtype == torch.bfloat16 else a[n]
        y = b[n].view(torch.uint8) if b[n].dtype == torch.bfloat16 else b[n]
        assert torch.equal(x, y), f"{what}: {n} differs from pv_prune_pipeline"


def test_noalloc_matches_workspace_call_on_shrinking_inputs():
    from paper_2608_25332_amd import provip
    # hi-res (35 MiB of scratch), then LLaVA-1.5 B=1 (4 MiB), then the tiny
    # fp32 workload: each call smaller than the one before
    for wid in (4, 2, 1):
        w = W.make_workload(wid)
        _say(f"[noalloc] workload {wid} ({w.spec.name}) B={w.spec.B} Nv={w.spec.Nv}")
        ins = _inputs(w)
        ref = provip.pv_prune_pipeline(*ins, w.heads, w.N1, w.N2)
        torch.cuda.synchronize()
        out = {n: torch.empty_like(ref[n]) for n in provip.PIPELINE_OUTPUTS}
        for t in out.values():
            t.view(torch.uint8).fill_(0xA5)
        before = torch.cuda.memory_allocated()
        provip.pv_prune_pipeline_noalloc(*ins, w.heads, w.N1, w.N2, out=out)
        torch.cuda.synchronize()
        assert torch.cuda.memory_allocated() == before
        _assert_same(out, ref, f"workload {wid}")


def test_noalloc_rejects_a_problem_larger_than_the_scratch():
    """16 samples of the 13B 8-frame shape need more than the static scratch:
    the call returns PV_ERR_SCRATCH and enqueues nothing."""
    from paper_2608_25332_amd import provip
    B, Nv, Nt, d, H, hd, nh, N1, N2 = 16, 4608, 128, 5120, 40, 128, 5, 1152, 512
    assert provip.pv_pipeline_workspace_bytes(B, Nv, Nt, d, H, hd, nh, N1, N2, 1) > \
        provip.PV_STATIC_SCRATCH_BYTES
    dev = "cuda:0"
    bf = torch.bfloat16
    vis = torch.zeros((B, Nv, d), dtype=bf, device=dev)
    anc = torch.zeros((B, Nt, d), dtype=bf, device=dev)
    q = torch.zeros((B, H, Nt, hd), dtype=bf, device=dev)
    kf = torch.zeros((B, H, Nv, hd), dtype=bf, device=dev)
    heads = np.tile(np.arange(nh, dtype=np.int32), (B, 1))
    shapes = {"kept1": ((B, N1), torch.int32), "score1": ((B, Nv), torch.float32),
              "assign": ((B, Nv), torch.int32), "merged": ((B, N1, d), bf),
              "k1": ((B, H, N1, hd), bf), "v1": ((B, H, N1, hd), bf),
              "kept2": ((B, N2), torch.int32), "score2": ((B, N1), torch.float32),
              "hidden2": ((B, N2, d), bf), "k2": ((B, H, N2, hd), bf),
              "v2": ((B, H, N2, hd), bf)}
    out = {n: torch.full(s, 7, dtype=t, device=dev) for n, (s, t) in shapes.items()}
    with pytest.raises(provip.ProvipError) as e:
        provip.pv_prune_pipeline_noalloc(vis, anc, q, kf, kf, heads, N1, N2, out=out)
    assert e.value.status == -9
    torch.cuda.synchronize()
    assert bool((out["kept1"] == 7).all()) and bool((out["kept2"] == 7).all())
