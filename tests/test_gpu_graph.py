"""The pruning step captured in a HIP graph: every replay, with eager work
and synchronisations in between, must reproduce the eager result bit for
bit (the library records no memset node and keeps no state between calls)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.mark.parametrize("form", ["one_stream", "two_streams", "shared_launches"])
def test_graph_replays_match_eager(form):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import bench
    from paper_2608_25332_amd import workloads as W

    dev = torch.device("cuda:0")
    w = W.make_workload(2)
    step = bench.Step(w, dev, form=form)
    step.run()
    torch.cuda.synchronize()
    ref = step.snapshot()
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        step.run()
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step.run()
    torch.cuda.synchronize()
    for i in range(5):
        # scribble over the outputs eagerly, then replay
        for t in (step.o1["kept"], step.o1["assign"], step.o2["kept"], step.hid2, step.k2):
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        snap = step.snapshot()
        for k in ref:
            assert torch.equal(ref[k], snap[k]), (i, k)
        step.run()   # eager work between replays
        torch.cuda.synchronize()
