"""Benchmark of the ProViP pruning hot path on one MI355X.

One step = the whole hot path over one batch of the LLaVA-1.5-7B-shaped
workload (B=1, 576 visual tokens, d=4096, 32 heads x 128, 64 text rows,
4 selected heads, N1=192, N2=64):

  1. pv_prune_dedup       cosine to the text anchors, centring, max-pool,
                          top-N1, pruned x kept Gram + argmax, merge
  2. pv_prune_gather x2   K and V rows of the N1 kept tokens (stands in for
                          the layers that would produce them)
  3. pv_prune_head_aware  head-subset softmax score + top-N2
  4. pv_prune_gather x3   hidden (merged), K and V rows of the N2 kept tokens

Inputs are seeded synthetic tensors already resident in HBM.  The timed
region replays the step captured as one HIP graph K times between two HIP
events (the step is launch-bound at this size).  A second, eager pass over
the same steps records a HIP event pair around every kernel (through the
*_timed entry points) for the per-kernel breakdown and the roofline of the
dominant kernel.  The CPU oracle is timed on a bounded sample of the same
workload on the host.

Prints one JSON line.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "pruning-op latency (us) + visual tokens/s at LLaVA-1.5-7B shape; % HBM/MFMA peak"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", type=int, default=2, help="workload id (2 = LLaVA-1.5-7B)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="budget of the CPU-oracle baseline leg (0 disables it)")
    ap.add_argument("--eager-steps", type=int, default=200)
    ap.add_argument("--no-graph", action="store_true")
    return ap.parse_args()


class Step:
    """Buffers and the kernel sequence of one step (all preallocated)."""

    def __init__(self, w, dev):
        import torch

        from paper_2608_25332_amd import provip
        self.torch = torch
        self.pv = provip
        self.lib = provip.load()
        s = w.spec
        self.w = w
        self.dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32

        def dev_t(a):
            from paper_2608_25332_amd import workloads as W
            if w.dtype == "bf16":
                return torch.from_numpy(W.bf16_bits(a).view(np.int16)).view(torch.bfloat16).to(dev)
            return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)

        self.vis, self.anc = dev_t(w.vis), dev_t(w.anchors)
        self.q, self.kf, self.vf = dev_t(w.q), dev_t(w.k_full), dev_t(w.v_full)
        self.heads = np.ascontiguousarray(w.heads, np.int32)
        B, Nv, d, H, hd, N1, N2 = s.B, s.Nv, s.d, s.H, s.hd, w.N1, w.N2
        i32, f32 = torch.int32, torch.float32
        self.o1 = {"kept": torch.empty((B, N1), dtype=i32, device=dev),
                   "score": torch.empty((B, Nv), dtype=f32, device=dev),
                   "assign": torch.empty((B, Nv), dtype=i32, device=dev),
                   "merged": torch.empty((B, N1, d), dtype=self.dt, device=dev)}
        self.o2 = {"kept": torch.empty((B, N2), dtype=i32, device=dev),
                   "score": torch.empty((B, N1), dtype=f32, device=dev)}
        self.k1 = torch.empty((B, H, N1, hd), dtype=self.dt, device=dev)
        self.v1 = torch.empty_like(self.k1)
        self.hid2 = torch.empty((B, N2, d), dtype=self.dt, device=dev)
        self.k2 = torch.empty((B, H, N2, hd), dtype=self.dt, device=dev)
        self.v2 = torch.empty_like(self.k2)
        code = 1 if w.dtype == "bf16" else 0
        self.ws1 = torch.empty(provip.pv_dedup_workspace_bytes(B, Nv, s.Nt, d, N1, code),
                               dtype=torch.uint8, device=dev)
        self.ws2 = torch.empty(provip.pv_head_aware_workspace_bytes(B, H, s.Nt, N1, hd,
                                                                    self.heads.shape[1], N2, code),
                               dtype=torch.uint8, device=dev)

    def run(self, ev=None):
        """Enqueue one step.  With ev (a list of torch events) every kernel is
        bracketed: returns the list of (name, start_event, end_event)."""
        pv = self.pv
        marks = []
        n1 = Step.DEDUP_EVENTS
        e1 = ev[:n1] if ev else None
        r = pv.pv_prune_dedup(self.vis, self.anc, self.w.N1, out=self.o1, workspace=self.ws1,
                              events=e1)
        if ev:
            for i, nm in enumerate(r["kernel_names"]):
                marks.append((nm, ev[i], ev[i + 1]))
        base = n1
        seq = [
            ("gather_kv1", lambda: pv.pv_prune_gather_batch([self.kf, self.vf], self.o1["kept"],
                                                            outs=[self.k1, self.v1])),
        ]
        for nm, fn in seq:
            if ev:
                ev[base].record()
            fn()
            if ev:
                ev[base + 1].record()
                marks.append((nm, ev[base], ev[base + 1]))
                base += 2
        e2 = ev[base:base + Step.HEAD_EVENTS] if ev else None
        h = pv.pv_prune_head_aware(self.q, self.k1, self.heads, self.w.N2, out=self.o2,
                                   workspace=self.ws2, events=e2)
        if ev:
            for i, nm in enumerate(h["kernel_names"]):
                marks.append((nm, ev[base + i], ev[base + i + 1]))
            base += Step.HEAD_EVENTS
        seq = [
            ("gather_hkv2", lambda: pv.pv_prune_gather_batch(
                [self.o1["merged"], self.k1, self.v1], self.o2["kept"],
                outs=[self.hid2, self.k2, self.v2])),
        ]
        for nm, fn in seq:
            if ev:
                ev[base].record()
            fn()
            if ev:
                ev[base + 1].record()
                marks.append((nm, ev[base], ev[base + 1]))
                base += 2
        return marks

    DEDUP_EVENTS = 8   # up to 7 kernels + 1
    HEAD_EVENTS = 4    # up to 3 kernels + 1
    N_EVENTS = DEDUP_EVENTS + 2 + HEAD_EVENTS + 2

    def snapshot(self):
        return {k: v.clone() for k, v in [("kept1", self.o1["kept"]), ("assign", self.o1["assign"]),
                                          ("merged", self.o1["merged"]), ("kept2", self.o2["kept"]),
                                          ("score2", self.o2["score"]), ("hid2", self.hid2),
                                          ("k2", self.k2), ("v2", self.v2)]}


DEDUP_KERNELS = ("cos_stream", "center", "select", "gram_stream", "gram_tile", "gram_finish",
                 "merge")


def algorithmic(w):
    """Algorithmic HBM bytes and flops per kernel per launch (one batch): the
    bytes a kernel must move at least (its inputs read once, its outputs
    written once) and the flops its step defines."""
    s = w.spec
    B, Nv, d, Nt, H, hd, N1, N2 = s.B, s.Nv, s.d, s.Nt, s.H, s.hd, w.N1, w.N2
    nh = w.heads.shape[1]
    e = 2 if w.dtype == "bf16" else 4
    Mp = Nv - N1
    gram = dict(bytes=B * Nv * d * e, flops=2.0 * B * Mp * N1 * d)
    return {
        # cosine: read the visual tokens and the anchors once, write M
        "cos_stream": dict(bytes=B * (Nv + Nt) * d * e + B * Nt * Nv * 4, flops=2.0 * B * Nt * Nv * d),
        # centring + max-pool: read M, write p
        "center": dict(bytes=B * (Nt * Nv + Nv) * 4, flops=2.0 * B * Nt * Nv),
        # top-N1: read p, write kept / pruned / slots
        "select": dict(bytes=B * Nv * 4 * 3, flops=0.0),
        # Gram: read every visual token once (pruned rows and kept rows)
        "gram_stream": gram, "gram_tile": gram,
        "gram_finish": dict(bytes=B * Mp * 4 * 2, flops=0.0),
        # merge: read every visual token once, write the N1 centroids
        "merge": dict(bytes=B * (Nv + N1) * d * e, flops=1.0 * B * Nv * d),
        # read + write the K and V rows of the N1 kept tokens
        "gather_kv1": dict(bytes=2 * 2 * B * H * N1 * hd * e, flops=0.0),
        # score: Q and K of the selected heads only
        "score_partial": dict(bytes=B * nh * (Nt + N1) * hd * e, flops=2.0 * 2 * B * nh * Nt * N1 * hd),
        "score_select": dict(bytes=B * N1 * 4, flops=0.0),
        # read + write the hidden, K and V rows of the N2 kept tokens
        "gather_hkv2": dict(bytes=2 * B * N2 * (d + 2 * H * hd) * e, flops=0.0),
    }


def graph_time_us(torch, fn, reps=300):
    """Average time of fn() captured once in a HIP graph and replayed reps
    times back to back between two events (no profiler attached)."""
    dev = torch.cuda.current_device()
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    for _ in range(10):
        g.replay()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    z = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        g.replay()
    z.record()
    torch.cuda.synchronize()
    return a.elapsed_time(z) * 1000.0 / reps


def stage_breakdown(torch, step):
    """Per-stage cost from graph replays of the public calls alone."""
    pv, w = step.pv, step.w
    o1 = step.o1
    cuts = {
        "dedup_kept_only": lambda: pv.pv_prune_dedup(step.vis, step.anc, w.N1, want_score=False,
                                                     want_assign=False, want_merged=False,
                                                     out=o1, workspace=step.ws1),
        "dedup_with_assign": lambda: pv.pv_prune_dedup(step.vis, step.anc, w.N1, want_merged=False,
                                                       out=o1, workspace=step.ws1),
        "dedup_full": lambda: pv.pv_prune_dedup(step.vis, step.anc, w.N1, out=o1, workspace=step.ws1),
        "gather_kv1": lambda: pv.pv_prune_gather_batch([step.kf, step.vf], o1["kept"],
                                                       outs=[step.k1, step.v1]),
        "head_aware": lambda: pv.pv_prune_head_aware(step.q, step.k1, step.heads, w.N2,
                                                     out=step.o2, workspace=step.ws2),
        "gather_hkv2": lambda: pv.pv_prune_gather_batch([o1["merged"], step.k1, step.v1],
                                                        step.o2["kept"],
                                                        outs=[step.hid2, step.k2, step.v2]),
    }
    return {k: graph_time_us(torch, f) for k, f in cuts.items()}


def cpu_baseline(w, seconds):
    """The CPU oracle, as it stands, over repeats of the same batch until the
    time budget is used (at least one full step)."""
    import oracle

    s = w.spec
    reps = 0
    t0 = time.perf_counter()
    while True:
        ref = oracle.dedup(w.anchors, w.vis, w.N1)
        kept1 = ref["kept"]
        k1 = np.stack([w.k_full[b][:, kept1[b]] for b in range(s.B)])
        v1 = np.stack([w.v_full[b][:, kept1[b]] for b in range(s.B)])
        kept2, _ = oracle.head_aware(w.q, k1, w.heads, w.N2)
        oracle.gather(ref["merged"], kept2)
        oracle.gather(k1, kept2)
        oracle.gather(v1, kept2)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    toks = reps * s.B * s.Nv
    return {"value": toks / el, "unit": "visual tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"{reps} full steps (dedup+merge, head-aware, gathers) of the {s.name} batch "
                      f"(B={s.B}, Nv={s.Nv}) in {el:.2f} s, single-threaded fp64 C oracle",
            "seconds": round(el, 3)}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "gpus_requested": args.gpus}))
        sys.exit(2)
    import torch

    from paper_2608_25332_amd import workloads as W

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = W.make_workload(args.workload)
    s = w.spec
    step = Step(w, dev)
    stream = torch.cuda.current_stream(dev)

    # eager reference outputs
    step.run()
    torch.cuda.synchronize()
    ref = step.snapshot()

    # ---- headline: graph replay
    use_graph = not args.no_graph
    graph = None
    if use_graph:
        side = torch.cuda.Stream(dev)
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            for _ in range(3):
                step.run()
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step.run()
        torch.cuda.synchronize()
        # every replay must reproduce the eager result
        for _ in range(3):
            graph.replay()
            torch.cuda.synchronize()
            snap = step.snapshot()
            for k in ref:
                if not torch.equal(ref[k], snap[k]):
                    raise RuntimeError(f"graph replay differs from eager in {k}")
            step.run()
            torch.cuda.synchronize()
    run_once = graph.replay if graph is not None else step.run
    for _ in range(args.warmup):
        run_once()
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record()
    for _ in range(args.steps):
        run_once()
    t_end.record()
    torch.cuda.synchronize()
    ms_total = t_start.elapsed_time(t_end)
    ms_per_step = ms_total / args.steps

    # ---- eager pass with an event pair around every kernel
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(Step.N_EVENTS)]
           for _ in range(args.eager_steps)]
    for row in evs:          # torch creates the HIP event on first record
        for e in row:
            e.record()
    torch.cuda.synchronize()
    all_marks = []
    e_start = torch.cuda.Event(enable_timing=True)
    e_end = torch.cuda.Event(enable_timing=True)
    e_start.record()
    for i in range(args.eager_steps):
        # keep the GPU behind the host so each event is stamped when the GPU
        # reaches it, not while it waits for the next launch
        torch.cuda._sleep(2_000_000)
        all_marks.append(step.run(evs[i]))
    e_end.record()
    torch.cuda.synchronize()
    per = {}
    for marks in all_marks:
        for nm, a, b in marks:
            per.setdefault(nm, []).append(a.elapsed_time(b) * 1000.0)
    kern_us = {k: float(np.mean(v)) for k, v in per.items()}
    kern_p50 = {k: float(np.median(v)) for k, v in per.items()}
    stage_us = {
        "dedup": sum(kern_us[k] for k in DEDUP_KERNELS if k in kern_us),
        "kv_of_kept": kern_us["gather_kv1"],
        "head_aware": kern_us["score_partial"] + kern_us["score_select"],
        "gather": kern_us["gather_hkv2"],
    }
    breakdown = stage_breakdown(torch, step)
    step.run()
    torch.cuda.synchronize()
    # last replay/eager output still matches
    snap = step.snapshot()
    for k in ref:
        if not torch.equal(ref[k], snap[k]):
            raise RuntimeError(f"benchmark output drifted in {k}")

    alg = algorithmic(w)
    dom = max(kern_us, key=lambda k: kern_us[k])
    a = alg[dom]
    sec = kern_us[dom] * 1e-6
    ai = a["flops"] / a["bytes"] if a["bytes"] else float("inf")
    ridge = BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    if ai >= ridge:
        roof = {"bound": "mfma", "achieved": a["flops"] / sec / 1e12, "peak": BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": a["bytes"] / sec / 1e9, "peak": HBM_PEAK_GBS,
                "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = None
    roof["kernel"] = dom
    roof["kernel_us"] = kern_us[dom]
    roof["algorithmic_bytes"] = a["bytes"]
    roof["algorithmic_flops"] = a["flops"]

    toks = s.B * s.Nv
    value = toks / (ms_per_step * 1e-3)
    line = {
        "metric": METRIC,
        "value": value,
        "unit": "visual tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": s.name, "B": s.B, "Nv": s.Nv, "d": s.d, "H": s.H, "hd": s.hd,
                   "Nt": s.Nt, "heads_per_sample": int(w.heads.shape[1]), "N1": w.N1, "N2": w.N2,
                   "timing": "hip-graph replay of the full step" if graph is not None else "eager"},
        "latency_us": {"pipeline": ms_per_step * 1000.0,
                       "pipeline_eager_evented": e_start.elapsed_time(e_end) * 1000.0 / args.eager_steps,
                       "stages_eager": stage_us, "kernels_eager_mean": kern_us,
                       "kernels_eager_p50": kern_p50,
                       "stages_graph_replay": breakdown},
        "roofline": roof,
    }
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
