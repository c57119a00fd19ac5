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
events (the step is launch-bound at this size).  Then every kernel of the
step is launched back to back between two HIP events on the library's
stream (the *_timed entry points with reps > 1) for its average duration,
which gives the per-kernel and per-stage roofline positions and the
roofline of the dominant kernel.  The step takes whichever of three forms
replays fastest: the four calls on one stream, the merge branch on a
second stream, or one pv_prune_pipeline call whose two chains after the
top-N1 share launches; the roofline line is taken over the kernels of the
form that is timed (pv_prune_pipeline_timed for the shared launches).  The
CPU oracle is timed on a bounded sample of the same workload on the host.

Prints one JSON line.
"""

from __future__ import annotations

import argparse
import json
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
    ap.add_argument("--kernel-reps", type=int, default=20,
                    help="back-to-back launches of each kernel per timing sample")
    ap.add_argument("--kernel-iters", type=int, default=10, help="timing samples per kernel")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--pmc-pass", action="store_true",
                    help="counter-collection pass: `steps` eager steps, then a copy kernel of "
                         "known size (--calib-mib) to scale the counters; no timing")
    ap.add_argument("--calib-mib", type=int, default=256)
    ap.add_argument("--split", action="store_true",
                    help="time the step with the merge branch on a second stream "
                         "(the same as --streams 2)")
    ap.add_argument("--streams", choices=["1", "2", "shared", "auto"], default="auto",
                    help="the step as four calls on one stream, with the merge branch on a "
                         "second stream, as one pv_prune_pipeline call (the two chains after "
                         "the top-N1 share launches), or whichever of the three replays fastest "
                         "(measured before the timed steps)")
    ap.add_argument("--cold-mib", type=int, default=640,
                    help="input copies rotated through for the cold-cache timing (0 disables it)")
    ap.add_argument("--per-config", default="3,4,5",
                    help="workload ids measured after the headline for the per_config block "
                         "(empty: none)")
    ap.add_argument("--gemm-calibration", action="store_true",
                    help="instead of the step: the pruned x kept Gram of the hi-res and 13B "
                         "workloads as a library GEMM (torch.bmm, i.e. hipBLASLt, on rows already "
                         "gathered) beside this library's gram_tile (rows gathered in the kernel, "
                         "argmax fused); prints its own JSON line")
    ap.add_argument("--score-sweep", action="store_true",
                    help="instead of the step: the head-aware call at the LLaVA-1.5-7B shape over "
                         "a batch sweep, with the selected heads and with all heads; prints its "
                         "own JSON line")
    return ap.parse_args()


class Step:
    """Buffers and the kernel sequence of one step (all preallocated)."""

    FORMS = ("one_stream", "two_streams", "shared_launches")

    def __init__(self, w, dev, form="one_stream"):
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
        self.wsp = torch.empty(provip.pv_pipeline_workspace_bytes(
            B, Nv, s.Nt, d, H, hd, self.heads.shape[1], N1, N2, code), dtype=torch.uint8,
            device=dev)
        self.pipe_out = {"kept1": self.o1["kept"], "score1": self.o1["score"],
                         "assign": self.o1["assign"], "merged": self.o1["merged"], "k1": self.k1,
                         "v1": self.v1, "kept2": self.o2["kept"], "score2": self.o2["score"],
                         "hidden2": self.hid2, "k2": self.k2, "v2": self.v2}
        # second stream (default priority) and the fork/join events of the
        # two-stream step; torch creates a HIP event on its first record
        assert form in self.FORMS
        self.form = form
        self.side = torch.cuda.Stream(dev)
        self.ev_sel = torch.cuda.Event()
        self.ev_done = torch.cuda.Event()
        self.ev_sel.record()
        self.ev_done.record()
        torch.cuda.synchronize()

    def gather_kv1(self):
        self.pv.pv_prune_gather_batch([self.kf, self.vf], self.o1["kept"], outs=[self.k1, self.v1])

    def gather_hkv2(self):
        self.pv.pv_prune_gather_batch([self.o1["merged"], self.k1, self.v1], self.o2["kept"],
                                      outs=[self.hid2, self.k2, self.v2])

    def run(self):
        """Enqueue one step on the current stream.  In the two-stream form the
        nearest-centroid and merge kernels run on a second stream, overlapped
        with the K/V gather and the head-aware score (they meet again before
        the final gather, which needs the merged rows).  In the shared-launch
        form the step is one pv_prune_pipeline call, whose two chains after
        the top-N1 share launches where the shapes allow it."""
        pv, w = self.pv, self.w
        if self.form == "shared_launches":
            pv.pv_prune_pipeline(self.vis, self.anc, self.q, self.kf, self.vf, self.heads, w.N1,
                                 w.N2, out=self.pipe_out, workspace=self.wsp)
        elif self.form == "two_streams":
            cur = self.torch.cuda.current_stream()
            pv.pv_prune_dedup(self.vis, self.anc, w.N1, out=self.o1, workspace=self.ws1,
                              split=(self.side, self.ev_sel, self.ev_done))
            self.gather_kv1()
            pv.pv_prune_head_aware(self.q, self.k1, self.heads, w.N2, out=self.o2,
                                   workspace=self.ws2)
            cur.wait_event(self.ev_done)
            self.gather_hkv2()
        else:
            pv.pv_prune_dedup(self.vis, self.anc, w.N1, out=self.o1, workspace=self.ws1)
            self.gather_kv1()
            pv.pv_prune_head_aware(self.q, self.k1, self.heads, w.N2, out=self.o2,
                                   workspace=self.ws2)
            self.gather_hkv2()

    DEDUP_EVENTS = 9   # up to 8 kernels + 1
    HEAD_EVENTS = 4    # up to 3 kernels + 1

    def snapshot(self):
        return {k: v.clone() for k, v in [("kept1", self.o1["kept"]), ("assign", self.o1["assign"]),
                                          ("merged", self.o1["merged"]), ("kept2", self.o2["kept"]),
                                          ("score2", self.o2["score"]), ("hid2", self.hid2),
                                          ("k2", self.k2), ("v2", self.v2)]}


# kernel -> the stage of the hot path it belongs to
STAGE_OF = {
    "cos_full": "cosine", "cos_partial": "cosine", "cos_reduce": "cosine", "center": "cosine",
    "select": "select", "gram_partial": "gram", "gram_reduce": "gram", "gram_tile": "gram",
    "gram_finish": "gram", "bucket": "merge", "merge": "merge", "gather_kv1": "kv_of_kept",
    "score_partial": "head_aware", "score_select": "head_aware", "gather_hkv2": "gather",
}


# kernel of the shared-launch step (pv_prune_pipeline_timed's name) -> the
# kernels of the separate step whose work it does
SHARED_PARTS = {"gram_partial+score_partial": ("gram_partial", "score_partial"),
                "gram_reduce+score_select+gather_kv1": ("gram_reduce", "score_select",
                                                        "gather_kv1"),
                "merge+gather_hkv2": ("merge", "gather_hkv2")}
# kernel name in bench.py -> the name rocprofv3 reports (without "_kernel" and
# template arguments), which keys the committed counter summaries
PROFILED_ALT = {"merge": ["merge_csr"], "cos_reduce": ["cos_reduce4"]}
PROFILED_NAME = {"gram_partial+score_partial": "gram_score",
                 "gram_reduce+score_select+gather_kv1": "reduce_select_gather",
                 "merge+gather_hkv2": "merge", "gather_kv1": "gather", "gather_hkv2": "gather"}


def algorithmic(w):
    """Algorithmic HBM bytes and flops per launch (one batch), per kernel and
    per stage: the bytes a step must move at least (its inputs read once,
    its outputs written once) and the flops it defines.  Split-k partial
    sums are an implementation choice and are not counted."""
    s = w.spec
    B, Nv, d, Nt, H, hd, N1, N2 = s.B, s.Nv, s.d, s.Nt, s.H, s.hd, w.N1, w.N2
    nh = w.heads.shape[1]
    e = 2 if w.dtype == "bf16" else 4
    Mp = Nv - N1
    gram_flops = 2.0 * B * Mp * N1 * d
    kern = {
        # cosine products: read the visual tokens and the anchors once
        "cos_partial": dict(bytes=B * (Nv + Nt) * d * e, flops=2.0 * B * Nt * Nv * d),
        # one-pass cosine: read the visual tokens and anchors, write M and norms
        "cos_full": dict(bytes=B * (Nv + Nt) * d * e + B * (Nt * Nv + Nv) * 4,
                         flops=2.0 * B * Nt * Nv * d),
        # cosines: write M and the inverse token norms
        "cos_reduce": dict(bytes=B * (Nt * Nv + Nv) * 4, flops=3.0 * B * Nt * Nv),
        # centring + max-pool: read M, write p
        "center": dict(bytes=B * (Nt * Nv + Nv) * 4, flops=2.0 * B * Nt * Nv),
        # top-N1: read p, write kept / pruned / slots
        "select": dict(bytes=B * Nv * 4 * 3, flops=0.0),
        # Gram: read every visual token once (pruned rows and kept rows)
        "gram_partial": dict(bytes=B * Nv * d * e, flops=gram_flops),
        "gram_tile": dict(bytes=B * Nv * d * e, flops=gram_flops),
        # argmax: read the inverse norms, write the assignment
        "gram_reduce": dict(bytes=B * Nv * 4 * 2, flops=1.0 * B * Mp * N1),
        "gram_finish": dict(bytes=B * Mp * 4 * 2, flops=0.0),
        # member lists: read the assignment, write the lists
        "bucket": dict(bytes=B * (Nv * 4 * 2 + N1 * 8), flops=0.0),
        # merge: read every visual token once, write the N1 centroids
        "merge": dict(bytes=B * (Nv + N1) * d * e, flops=1.0 * B * Nv * d),
        # read + write the K and V rows of the N1 kept tokens
        "gather_kv1": dict(bytes=2 * 2 * B * H * N1 * hd * e, flops=0.0),
        # score: Q and K of the selected heads only
        "score_partial": dict(bytes=B * nh * (Nt + N1) * hd * e,
                              flops=2.0 * 2 * B * nh * Nt * N1 * hd),
        "score_select": dict(bytes=B * N1 * 4 * 2, flops=0.0),
        # read + write the hidden, K and V rows of the N2 kept tokens
        "gather_hkv2": dict(bytes=2 * B * N2 * (d + 2 * H * hd) * e, flops=0.0),
    }
    # kernels of the shared-launch step: each does the work of its parts
    for parts in SHARED_PARTS.values():
        kern["+".join(parts)] = dict(bytes=sum(kern[p]["bytes"] for p in parts),
                                     flops=sum(kern[p]["flops"] for p in parts))
    # the merge writes the kept slots' rows to their compacted places itself:
    # the compaction reads no merged row
    kern["merge+gather_hkv2"]["bytes"] -= B * N2 * d * e
    stage = {
        "cosine": dict(bytes=B * (Nv + Nt) * d * e + B * Nv * 4, flops=2.0 * B * Nt * Nv * d),
        "select": kern["select"],
        "gram": dict(bytes=B * Nv * d * e + B * Nv * 4, flops=gram_flops),
        "merge": kern["merge"],
        "kv_of_kept": kern["gather_kv1"],
        "head_aware": dict(bytes=B * nh * (Nt + N1) * hd * e + B * N2 * 4,
                           flops=kern["score_partial"]["flops"]),
        "gather": kern["gather_hkv2"],
    }
    return kern, stage


def roof(a, sec):
    """Roofline position of work a (bytes, flops) done in sec seconds: bound
    by MFMA when its arithmetic intensity is above the bf16 ridge, else HBM."""
    ridge = BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    ai = a["flops"] / a["bytes"] if a["bytes"] else float("inf")
    if ai >= ridge:
        r = {"bound": "mfma", "achieved": a["flops"] / sec / 1e12, "peak": BF16_PEAK_TFLOPS,
             "unit": "TFLOP/s"}
    else:
        r = {"bound": "hbm", "achieved": a["bytes"] / sec / 1e9, "peak": HBM_PEAK_GBS,
             "unit": "GB/s"}
    r["frac"] = r["achieved"] / r["peak"]
    return r


def sleep_cycles_for(torch, ms):
    """Argument of torch.cuda._sleep that keeps the GPU busy for about ms."""
    a = torch.cuda.Event(enable_timing=True)
    z = torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(1000)
    a.record()
    torch.cuda._sleep(1_000_000)
    z.record()
    torch.cuda.synchronize()
    per_ms = 1_000_000 / max(a.elapsed_time(z), 1e-3)
    return int(per_ms * ms)


def kernel_times(torch, step, reps, iters):
    """Average duration of every kernel of the step: the kernels of each call
    are launched reps times back to back between two HIP events recorded on
    the stream the library launches on (the current stream).  A spin kernel
    queued first keeps the GPU behind the host, so the launches run back to
    back rather than at the host's pace; a sample whose spin had already
    ended when the host finished enqueuing is taken again with a longer
    spin."""
    pv = step.pv
    per = {}
    hold_ms = 4.0
    done = 0
    while done < iters:
        e1 = [torch.cuda.Event(enable_timing=True) for _ in range(Step.DEDUP_EVENTS)]
        e2 = [torch.cuda.Event(enable_timing=True) for _ in range(Step.HEAD_EVENTS)]
        g1 = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        g2 = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        spun = torch.cuda.Event()
        for e in e1 + e2 + g1 + g2 + [spun]:  # torch creates the HIP event on first record
            e.record()
        torch.cuda.synchronize()
        torch.cuda._sleep(sleep_cycles_for(torch, hold_ms))
        spun.record()
        r1 = pv.pv_prune_dedup(step.vis, step.anc, step.w.N1, out=step.o1, workspace=step.ws1,
                               events=e1, reps=reps)
        g1[0].record()
        for _ in range(reps):
            step.gather_kv1()
        g1[1].record()
        r2 = pv.pv_prune_head_aware(step.q, step.k1, step.heads, step.w.N2, out=step.o2,
                                    workspace=step.ws2, events=e2, reps=reps)
        g2[0].record()
        for _ in range(reps):
            step.gather_hkv2()
        g2[1].record()
        starved = spun.query()
        torch.cuda.synchronize()
        if starved:
            hold_ms *= 2
            if hold_ms > 1000:
                raise RuntimeError("host cannot keep ahead of the GPU for the kernel timing")
            continue
        done += 1
        marks = [(nm, e1[i], e1[i + 1]) for i, nm in enumerate(r1["kernel_names"])]
        marks += [("gather_kv1", g1[0], g1[1])]
        marks += [(nm, e2[i], e2[i + 1]) for i, nm in enumerate(r2["kernel_names"])]
        marks += [("gather_hkv2", g2[0], g2[1])]
        for nm, a, b in marks:
            per.setdefault(nm, []).append(a.elapsed_time(b) * 1000.0 / reps)
    return {k: float(np.median(v)) for k, v in per.items()}


def shared_kernel_times(torch, step, reps, iters):
    """kernel_times for the shared-launch step (pv_prune_pipeline_timed):
    every launch of the one call repeated reps times back to back between
    two HIP events.  Empty when the shapes give no shared launches."""
    pv, w = step.pv, step.w
    per = {}
    hold_ms = 4.0
    done = 0
    while done < iters:
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(10)]
        spun = torch.cuda.Event()
        for e in ev + [spun]:
            e.record()
        torch.cuda.synchronize()
        torch.cuda._sleep(sleep_cycles_for(torch, hold_ms))
        spun.record()
        r = pv.pv_prune_pipeline(step.vis, step.anc, step.q, step.kf, step.vf, step.heads, w.N1,
                                 w.N2, out=step.pipe_out, workspace=step.wsp, events=ev,
                                 reps=reps)
        starved = spun.query()
        torch.cuda.synchronize()
        if r["n_kernels"] == 0:
            return {}
        if starved:
            hold_ms *= 2
            if hold_ms > 1000:
                raise RuntimeError("host cannot keep ahead of the GPU for the kernel timing")
            continue
        done += 1
        for i, nm in enumerate(r["kernel_names"]):
            per.setdefault(nm, []).append(ev[i].elapsed_time(ev[i + 1]) * 1000.0 / reps)
    return {k: float(np.median(v)) for k, v in per.items()}


def csrc_digest():
    """Digest of the library sources: counter figures taken from a build with
    another digest no longer describe the kernels."""
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2608_25332_amd", "csrc")
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".h")):
            h.update(f.encode())
            with open(os.path.join(d, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()[:16]


def load_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed PMC summary of this
    workload (FETCH_SIZE and WRITE_SIZE, scaled by a copy kernel of known
    size), or None when there is none or the sources changed since."""
    path = os.path.join(ROOT, "profiles", f"pmc_{workload}.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    i = txt.find("```json")
    if i < 0:
        return None
    j = txt.find("```", i + 7)
    try:
        rec = json.loads(txt[i + 7:j])
    except ValueError:
        return None
    if rec.get("csrc_digest") != csrc_digest():
        return None
    kernels = rec.get("kernels", {})
    # the same call runs another kernel at some shapes (member-list merge,
    # four-token slice reduction)
    names = [PROFILED_NAME.get(kernel, kernel)] + PROFILED_ALT.get(kernel, [])
    k = next((kernels[n] for n in names if n in kernels), None)
    if not k:
        return None
    return float(k["fetch_bytes"]) + float(k["write_bytes"])


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


def replay_percentiles(torch, fn_replay, reps=400):
    """p10 / p50 / p90 (us) of single replays, each between its own pair of
    HIP events (consecutive replays, so each still follows the previous one
    as in the timed loop)."""
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for a, z in ev:
        a.record()
        fn_replay()
        z.record()
    torch.cuda.synchronize()
    t = np.array([a.elapsed_time(z) * 1000.0 for a, z in ev])
    return {"p10": float(np.percentile(t, 10)), "p50": float(np.percentile(t, 50)),
            "p90": float(np.percentile(t, 90))}


def cold_times(torch, step, dev, budget_mib, rounds=6):
    """Step and dedup-call time with cold caches: enough copies of the step's
    inputs (visual tokens, anchors, Q, K and V of all tokens) that one
    rotation through them moves more than budget_mib, which is above the
    256 MB MALL and the L2s, so every replay finds its inputs in HBM only.
    One graph per copy; the replays go round robin."""
    names = ("vis", "anc", "q", "kf", "vf")
    orig = {n: getattr(step, n) for n in names}
    per_copy = sum(t.numel() * t.element_size() for t in orig.values())
    ncopy = max(2, -(-(budget_mib << 20) // per_copy))
    copies = [{n: t.clone() for n, t in orig.items()} for _ in range(ncopy)]
    stream = torch.cuda.current_stream(dev)
    pv, w = step.pv, step.w

    def capture(fn):
        side = torch.cuda.Stream(dev)
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            fn()
        stream.wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        return g

    g_step, g_dedup = [], []
    try:
        for c in copies:
            for n in names:
                setattr(step, n, c[n])
            g_step.append(capture(step.run))
            g_dedup.append(capture(lambda: pv.pv_prune_dedup(step.vis, step.anc, w.N1, out=step.o1,
                                                             workspace=step.ws1)))
    finally:
        for n in names:
            setattr(step, n, orig[n])
    torch.cuda.synchronize()
    out = {"input_copies": ncopy, "rotation_mib": round(ncopy * per_copy / 2**20, 1)}
    for key, gs in (("step", g_step), ("dedup_full", g_dedup)):
        for g in gs:
            g.replay()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        z = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(rounds):
            for g in gs:
                g.replay()
        z.record()
        torch.cuda.synchronize()
        out[key] = a.elapsed_time(z) * 1000.0 / (rounds * len(gs))
    del g_step, g_dedup, copies
    torch.cuda.synchronize()
    return out


def score_sweep(torch, dev):
    """Head-aware call at the LLaVA-1.5-7B shape (32 heads x 128, 64 text
    rows, 192 kept keys, keep 64) over B = 1 .. 256, with 4 selected heads
    per sample and with all 32 heads (host head lists), and with all heads
    from a device list at B = 64 .. 256.  Per point: the call's time from graph
    replays, the score kernel's average duration from back-to-back launches
    between HIP events, and the kernel's algorithmic HBM bytes (Q and K of
    the heads read) over that duration."""
    from paper_2608_25332_amd import provip as pv

    H, Nt, N, hd, N2 = 32, 64, 192, 128, 64
    Bmax = 256
    gen = torch.Generator(device=dev)
    gen.manual_seed(2)
    q_all = torch.randn((Bmax, H, Nt, hd), generator=gen, device=dev).to(torch.bfloat16)
    k_all = torch.randn((Bmax, H, N, hd), generator=gen, device=dev).to(torch.bfloat16)
    rng = np.random.default_rng(2)
    rows = []
    # host head lists at every point; device lists (one launch whatever the
    # batch) where a host list would take several launches or nearly so
    points = [(nh, B, False) for nh in (4, H) for B in (1, 4, 16, 64, 256)]
    points += [(H, B, True) for B in (64, 128, 256)]
    for nh, B, on_dev in points:
        q, k = q_all[:B], k_all[:B]
        heads = np.stack([rng.permutation(H)[:nh] for _ in range(B)]).astype(np.int32)
        if on_dev:
            heads = torch.from_numpy(heads).to(dev)
        out = {"kept": torch.empty((B, N2), dtype=torch.int32, device=dev),
               "score": torch.empty((B, N), dtype=torch.float32, device=dev)}
        ws = torch.empty(pv.pv_head_aware_workspace_bytes(B, H, Nt, N, hd, nh, N2, 1),
                         dtype=torch.uint8, device=dev)
        call = lambda: pv.pv_prune_head_aware(q, k, heads, N2, out=out, workspace=ws)
        call_us = graph_time_us(torch, call, reps=200)
        reps = 20
        samples = []
        for _ in range(5):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(Step.HEAD_EVENTS)]
            for e in ev:
                e.record()
            r = pv.pv_prune_head_aware(q, k, heads, N2, out=out, workspace=ws, events=ev,
                                       reps=reps)
            torch.cuda.synchronize()
            i = r["kernel_names"].index("score_partial")
            samples.append(ev[i].elapsed_time(ev[i + 1]) * 1000.0 / reps)
        kus = float(np.median(samples))
        nbytes = B * nh * (Nt + N) * hd * 2
        gbs = nbytes / (kus * 1e-6) / 1e9
        rows.append({"B": B, "heads_per_sample": nh, "heads_on_device": on_dev,
                     "call_us": call_us, "score_kernel_us": kus, "algorithmic_bytes": nbytes,
                     "achieved_GBs": gbs, "frac_hbm": gbs / HBM_PEAK_GBS})
        print(f"[score-sweep] B={B} heads={nh}{' (device list)' if on_dev else ''} "
              f"call {call_us:.2f} us, kernel {kus:.2f} us, {gbs:.0f} GB/s", file=sys.stderr,
              flush=True)
        del out, ws
    return {"score_sweep": rows, "shape": {"H": H, "Nt": Nt, "N": N, "hd": hd, "N2": N2,
                                           "dtype": "bf16"},
            "note": "warm caches; at B=256 with all heads the call reads 537 MB",
            "csrc_digest": csrc_digest()}


def measured_peaks(torch, dev):
    """The two published peaks the rooflines divide by, re-measured on this
    device (the fractions in this line stay against the published figures):
    HBM as the rate of the runtime's device copy of 1 GiB (bytes read +
    bytes written over the copy's time), and bf16 matrix throughput as the
    rate of the vendor GEMM (torch.matmul) on 8192^3, each the best of a few
    back-to-back batches between HIP events."""
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    ka = torch.randn((8192, 8192), device=dev).to(torch.bfloat16)
    kb = torch.randn((8192, 8192), device=dev).to(torch.bfloat16)
    kc = torch.matmul(ka, kb)
    torch.cuda.synchronize()

    def best_ms(fn, reps, tries=5):
        best = float("inf")
        for _ in range(tries):
            a = torch.cuda.Event(enable_timing=True)
            z = torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                fn()
            z.record()
            torch.cuda.synchronize()
            best = min(best, a.elapsed_time(z) / reps)
        return best

    copy_ms = best_ms(lambda: dst.copy_(src), 10)
    gemm_ms = best_ms(lambda: torch.matmul(ka, kb, out=kc), 5)
    hbm = 2.0 * n / (copy_ms * 1e-3) / 1e9
    tflops = 2.0 * 8192 ** 3 / (gemm_ms * 1e-3) / 1e12
    del src, dst, ka, kb, kc
    torch.cuda.synchronize()
    return {"hbm_copy_GBs": hbm, "hbm_copy_frac_of_published": hbm / HBM_PEAK_GBS,
            "bf16_gemm_8192_TFLOPs": tflops,
            "bf16_gemm_frac_of_published": tflops / BF16_PEAK_TFLOPS,
            "published": {"hbm_GBs": HBM_PEAK_GBS, "bf16_TFLOPs": BF16_PEAK_TFLOPS},
            "note": "rooflines use the published peaks; these are the device copy and the "
                    "vendor GEMM on this box"}


def gemm_calibration(torch, dev):
    """The Gram stage's contraction at the hi-res and 13B shapes (pruned x
    kept rows, 2 d (N_v - N_1) N_1 flops per sample) done two ways on the
    same device: torch.bmm on bf16 rows already gathered into contiguous
    [B, N_v - N_1, d] and [B, d, N_1] operands (the vendor GEMM library), and
    the dedup call's gram_tile kernel (rows gathered through index lists in
    the kernel, the row argmax fused), each timed back to back between HIP
    events.  A reference point for the MFMA fraction the Gram reaches."""
    from paper_2608_25332_amd import provip as pv
    from paper_2608_25332_amd import workloads as W

    rows = []
    for wid in (4, 5):
        w = W.make_workload(wid, with_kv=False)
        s = w.spec
        Mp, N1, d = s.Nv - w.N1, w.N1, s.d
        flops = 2.0 * s.B * Mp * N1 * d
        g = torch.Generator(device=dev)
        g.manual_seed(wid)
        A = torch.randn((s.B, Mp, d), generator=g, device=dev).to(torch.bfloat16)
        Bt = torch.randn((s.B, d, N1), generator=g, device=dev).to(torch.bfloat16).contiguous()

        def t_bmm():
            torch.bmm(A, Bt)
        t_bmm()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        z = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(20):
            t_bmm()
        z.record()
        torch.cuda.synchronize()
        bmm_us = a.elapsed_time(z) * 1000.0 / 20
        # this library's gram_tile in the dedup call (the kernel's own events)
        vis = torch.from_numpy(W.bf16_bits(w.vis).view(np.int16)).view(torch.bfloat16).to(dev)
        anc = torch.from_numpy(W.bf16_bits(w.anchors).view(np.int16)).view(torch.bfloat16).to(dev)
        out = pv.pv_prune_dedup(vis, anc, w.N1, want_merged=False)
        ws = out["workspace"]
        samples = []
        for _ in range(5):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(Step.DEDUP_EVENTS)]
            for e in ev:
                e.record()
            r = pv.pv_prune_dedup(vis, anc, w.N1, want_merged=False, out=out, workspace=ws,
                                  events=ev, reps=20)
            torch.cuda.synchronize()
            i = r["kernel_names"].index("gram_tile")
            samples.append(ev[i].elapsed_time(ev[i + 1]) * 1000.0 / 20)
        gt_us = float(np.median(samples))
        rows.append({"workload": s.name, "B": s.B, "M": Mp, "N": N1, "K": d, "flops": flops,
                     "torch_bmm_us": bmm_us,
                     "torch_bmm_frac_bf16_peak": flops / (bmm_us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS,
                     "gram_tile_us": gt_us,
                     "gram_tile_frac_bf16_peak": flops / (gt_us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS})
        print(f"[gemm-calibration] {s.name}: torch.bmm {bmm_us:.1f} us, gram_tile {gt_us:.1f} us",
              file=sys.stderr, flush=True)
        del A, Bt, vis, anc, out, ws
    return {"gemm_calibration": rows, "torch": torch.__version__,
            "note": "torch.bmm on contiguous bf16 operands (rows already gathered); gram_tile "
                    "gathers its rows through index lists and fuses the row argmax",
            "csrc_digest": csrc_digest()}


def visual_heads_timing(torch, step, n_vis=6):
    """Visual-head identification (all H heads of the N1 kept keys, the
    paper's N_vis = 6) at the step's shape: the call from graph replays and
    the confidence kernel's average duration between HIP events, with its
    roofline position (all heads of Q and K are read once)."""
    pv, w = step.pv, step.w
    s = w.spec
    B, H, Nt, N1, hd = s.B, s.H, s.Nt, w.N1, s.hd
    n_vis = min(n_vis, H)
    dev = step.q.device
    out = {"heads": torch.empty((B, n_vis), dtype=torch.int32, device=dev),
           "conf": torch.empty((B, H), dtype=torch.float32, device=dev)}
    ws = torch.empty(pv.pv_visual_heads_workspace_bytes(B, H, Nt), dtype=torch.uint8, device=dev)
    call = lambda: pv.pv_visual_heads(step.q, step.k1, n_vis, out=out, workspace=ws)
    call_us = graph_time_us(torch, call)
    reps, samples = 20, []
    for _ in range(5):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        for e in ev:
            e.record()
        r = pv.pv_visual_heads(step.q, step.k1, n_vis, out=out, workspace=ws, events=ev, reps=reps)
        torch.cuda.synchronize()
        i = r["kernel_names"].index("head_conf")
        samples.append(ev[i].elapsed_time(ev[i + 1]) * 1000.0 / reps)
    kus = float(np.median(samples))
    e = 2 if w.dtype == "bf16" else 4
    a = {"bytes": B * H * (Nt + N1) * hd * e, "flops": 2.0 * B * H * Nt * N1 * hd}
    rf = roof(a, kus * 1e-6)
    return {"n_vis": n_vis, "call_us": call_us, "head_conf_us": kus,
            "roofline": {"bound": rf["bound"], "achieved": rf["achieved"], "unit": rf["unit"],
                         "frac": rf["frac"], "algorithmic_bytes": a["bytes"]}}


def critical_text_timing(torch, step):
    """Critical text selection over the step's text rows (the anchors): the
    call from graph replays and the kernels' average durations."""
    pv, w = step.pv, step.w
    s = w.spec
    dev = step.anc.device
    out = {"mask": torch.empty((s.B, s.Nt), dtype=torch.int32, device=dev),
           "count": torch.empty((s.B,), dtype=torch.int32, device=dev),
           "r": torch.empty((s.B, s.Nt), dtype=torch.float32, device=dev)}
    code = 1 if w.dtype == "bf16" else 0
    ws = torch.empty(pv.pv_critical_text_workspace_bytes(s.B, s.Nt, s.d, code), dtype=torch.uint8,
                     device=dev)
    call = lambda: pv.pv_critical_text(step.anc, out=out, workspace=ws)
    call_us = graph_time_us(torch, call)
    reps, per = 20, {}
    for _ in range(5):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        for e in ev:
            e.record()
        r = pv.pv_critical_text(step.anc, out=out, workspace=ws, events=ev, reps=reps)
        torch.cuda.synchronize()
        for i, nm in enumerate(r["kernel_names"]):
            per.setdefault(nm, []).append(ev[i].elapsed_time(ev[i + 1]) * 1000.0 / reps)
    return {"call_us": call_us, "kernels_us": {k: float(np.median(v)) for k, v in per.items()}}


def progressive_timing(torch, w, dev):
    """The progressive schedule (pv_prune_progressive: critical text ->
    pruning before the LLM on the critical rows -> visual heads and
    head-aware pruning at the shallow layer -> all-head pruning at the middle
    layer) at the workload's shape, with a second seeded projection standing
    in for the middle layer: the call from graph replays, and visual tokens
    per second over it."""
    from paper_2608_25332_amd import provip as pv
    from paper_2608_25332_amd import workloads as W

    q_m, k_m = W.make_middle_layer(w)
    N1, n_vis, N2, N3 = W.progressive_budgets(w.spec)

    def dev_t(a):
        if w.dtype == "bf16":
            return torch.from_numpy(W.bf16_bits(a).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)

    ins = [dev_t(a) for a in (w.anchors, w.vis, w.q, w.k_full, q_m, k_m)]
    o = pv.pv_prune_progressive(*ins, N1, n_vis, N2, N3)
    ws = o.pop("workspace")
    call = lambda: pv.pv_prune_progressive(*ins, N1, n_vis, N2, N3, out=o, workspace=ws)
    us = graph_time_us(torch, call, reps=300)
    s = w.spec
    return {"call_us": us, "value": s.B * s.Nv / (us * 1e-6), "unit": "visual tokens/s",
            "budgets": {"N1": N1, "n_vis": n_vis, "N2": N2, "N3": N3},
            "note": "critical text, masked dedup with merge, visual heads + head-aware at a "
                    "shallow layer, all-head pruning at a middle layer (synthetic per-layer "
                    "Q/K), compactions between; one HIP graph"}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_step(w, b0: int, b1: int):
    """One full step of the oracle over samples [b0, b1) of the batch: dedup
    with the merge, the K/V rows of the kept tokens, head-aware, gathers.
    Returns the seconds of (dedup, head_aware, gather)."""
    import oracle

    s = w.spec
    a = time.perf_counter()
    ref = oracle.dedup(w.anchors[b0:b1], w.vis[b0:b1], w.N1)
    kept1 = ref["kept"]
    b = time.perf_counter()
    k1 = np.stack([w.k_full[b0 + i][:, kept1[i]] for i in range(b1 - b0)])
    v1 = np.stack([w.v_full[b0 + i][:, kept1[i]] for i in range(b1 - b0)])
    c = time.perf_counter()
    kept2, _ = oracle.head_aware(w.q[b0:b1], k1, w.heads[b0:b1], w.N2)
    d = time.perf_counter()
    oracle.gather(ref["merged"], kept2)
    oracle.gather(k1, kept2)
    oracle.gather(v1, kept2)
    e = time.perf_counter()
    del s
    return (b - a, d - c, (c - b) + (e - d))


def cpu_baseline(w, seconds):
    """The CPU oracle, as it stands, over repeats of the same batch until the
    time budget is used (at least one full step): first on one thread, then
    with every host CPU (up to 16) running whole steps at once.  The figure
    reported is the all-cores one; the one-thread figure and the seconds per
    stage are kept beside it."""
    from oracle.parallel import workers

    s = w.spec
    reps = 0
    st = [0.0, 0.0, 0.0]
    t0 = time.perf_counter()
    while True:
        for i, x in enumerate(_oracle_step(w, 0, s.B)):
            st[i] += x
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds / 2:
            break
    single = reps * s.B * s.Nv / el
    # all cores: every thread runs whole steps of the batch (ctypes releases
    # the GIL inside the oracle's C functions)
    import threading

    n = workers()
    done = [0] * n
    deadline = time.perf_counter() + seconds / 2

    def worker(i):
        while True:
            _oracle_step(w, 0, s.B)
            done[i] += 1
            if time.perf_counter() >= deadline:
                return

    t1 = time.perf_counter()
    th = [threading.Thread(target=worker, args=(i,)) for i in range(n)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    el_all = time.perf_counter() - t1
    steps_all = sum(done)
    value = steps_all * s.B * s.Nv / el_all
    return {"value": value, "unit": "visual tokens/s", "cores": n, "kind": "oracle",
            "sample": f"{steps_all} full steps (dedup+merge, head-aware, gathers) of the {s.name} "
                      f"batch (B={s.B}, Nv={s.Nv}) in {el_all:.2f} s, {n} threads each running "
                      f"whole steps of the fp64 C oracle",
            "seconds": round(el_all, 3),
            "single_thread": {"value": single, "cores": 1, "steps": reps,
                              "seconds": round(el, 3),
                              "seconds_per_step_by_stage": {
                                  k: round(v / reps, 4)
                                  for k, v in zip(("dedup", "head_aware", "gather"), st)}},
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count()}


def cpu_baseline_one_sample(w):
    """A bounded sample of a large workload: sample 0 of the batch, one full
    step of the oracle with the row ranges of its two big products (the
    cosine to the anchors, the nearest kept token of every row) spread over
    every host CPU (up to 16).  Visual tokens/s = Nv over its seconds."""
    import oracle
    from oracle.parallel import oracle_assign, oracle_p, workers

    s = w.spec
    t0 = time.perf_counter()
    p = oracle_p(w.anchors[:1], w.vis[:1])[0]
    kept1 = oracle.topk(p, w.N1)
    asg, _, _ = oracle_assign(w.vis[0], kept1, np.arange(s.Nv, dtype=np.int32))
    merged = oracle.merge(w.vis[0], kept1, asg)
    k1 = w.k_full[0][:, kept1][None]
    v1 = w.v_full[0][:, kept1][None]
    kept2, _ = oracle.head_aware(w.q[:1], k1, w.heads[:1], w.N2)
    oracle.gather(merged[None], kept2)
    oracle.gather(k1, kept2)
    oracle.gather(v1, kept2)
    el = time.perf_counter() - t0
    return {"value": s.Nv / el, "unit": "visual tokens/s", "cores": workers(), "kind": "oracle",
            "sample": f"sample 0 of the {s.name} batch (Nv={s.Nv}), one full step in {el:.2f} s, "
                      f"row ranges of the cosine and nearest-centroid products over "
                      f"{workers()} threads",
            "seconds": round(el, 3)}


def prepare(w, dev, args):
    """A Step in the form that replays fastest (unless one is forced)."""
    import torch

    first = {"1": "one_stream", "2": "two_streams", "shared": "shared_launches",
             "auto": "one_stream"}[args.streams]
    step = Step(w, dev, form="two_streams" if args.split else first)
    step.run()
    torch.cuda.synchronize()
    ref = step.snapshot()
    mode_us = {}
    if args.streams == "auto" and not args.split and not args.pmc_pass and not args.no_graph:
        for f in Step.FORMS:
            step.form = f
            mode_us[f] = graph_time_us(torch, step.run, reps=300)
        step.form = min(mode_us, key=lambda f: mode_us[f])
        torch.cuda.synchronize()
    return step, ref, mode_us


def capture_step(torch, step, dev, ref):
    """The step captured as one HIP graph; every replay must reproduce the
    eager result."""
    stream = torch.cuda.current_stream(dev)
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
    for _ in range(3):
        graph.replay()
        torch.cuda.synchronize()
        snap = step.snapshot()
        for k in ref:
            if not torch.equal(ref[k], snap[k]):
                raise RuntimeError(f"graph replay differs from eager in {k}")
        step.run()
        torch.cuda.synchronize()
    return graph


def timed_steps(torch, run_once, steps, warmup):
    for _ in range(warmup):
        run_once()
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record()
    for _ in range(steps):
        run_once()
    t_end.record()
    torch.cuda.synchronize()
    return t_start.elapsed_time(t_end) / steps


def rooflines(w, form, kern_us, shared_us):
    """Roofline of every kernel and stage, and of the dominant kernel of the
    form that is timed (with its HBM traffic from the committed counter
    summary when that matches the sources)."""
    alg_k, alg_s = algorithmic(w)
    kernels = {}
    for k, us in kern_us.items():
        r = roof(alg_k[k], us * 1e-6)
        kernels[k] = {"us": us, "bound": r["bound"], "achieved": r["achieved"], "unit": r["unit"],
                      "frac": r["frac"]}
        if alg_k[k]["flops"] > 0 and k.startswith("gram"):
            # the Gram against the matrix cores whatever its bound
            kernels[k]["frac_of_bf16_mfma_peak"] = alg_k[k]["flops"] / (us * 1e-6) / 1e12 / \
                BF16_PEAK_TFLOPS
    stage_us = {}
    for k, us in kern_us.items():
        stage_us[STAGE_OF[k]] = stage_us.get(STAGE_OF[k], 0.0) + us
    stages = {}
    for st_name, us in stage_us.items():
        r = roof(alg_s[st_name], us * 1e-6)
        stages[st_name] = {"us": us, "bound": r["bound"], "achieved": r["achieved"],
                           "unit": r["unit"], "frac": r["frac"]}
    shared = {}
    for k, us in shared_us.items():
        r = roof(alg_k[k], us * 1e-6)
        shared[k] = {"us": us, "bound": r["bound"], "achieved": r["achieved"], "unit": r["unit"],
                     "frac": r["frac"]}
    step_us = shared_us if form == "shared_launches" and shared_us else kern_us
    dom = max(step_us, key=lambda k: step_us[k])
    a = alg_k[dom]
    rf = roof(a, step_us[dom] * 1e-6)
    rf.update({"traffic": load_traffic(w.spec.name, dom), "kernel": dom,
               "kernel_us": step_us[dom], "algorithmic_bytes": a["bytes"],
               "algorithmic_flops": a["flops"]})
    return rf, kernels, stages, shared, stage_us


def config_of(w, form, split, graph):
    s = w.spec
    return {"workload": s.name, "B": s.B, "Nv": s.Nv, "d": s.d, "H": s.H, "hd": s.hd,
            "Nt": s.Nt, "heads_per_sample": int(w.heads.shape[1]), "N1": w.N1, "N2": w.N2,
            "streams": 2 if split else 1, "step_form": form,
            "timing": ("hip-graph replay of the full step" +
                       {"one_stream": "", "two_streams": ", merge branch on a second stream",
                        "shared_launches": ", one pv_prune_pipeline call (shared launches)"}[form]
                       if graph is not None else "eager")}


def measure_other(torch, wid, dev, args):
    """One of the larger workloads, for the per_config block: the step's
    graph-replay time in its fastest form, every kernel's duration and
    roofline, the per-stage roofline and a bounded CPU-oracle sample."""
    from paper_2608_25332_amd import workloads as W

    t0 = time.perf_counter()
    w = W.make_workload(wid)
    step, ref, mode_us = prepare(w, dev, args)
    graph = capture_step(torch, step, dev, ref)
    steps = max(20, min(args.steps, int(2e5 / max(min(mode_us.values()) if mode_us else 200, 1))))
    ms = timed_steps(torch, graph.replay, steps, max(5, args.warmup // 10))
    kern_us = kernel_times(torch, step, args.kernel_reps, max(3, args.kernel_iters // 2))
    shared_us = shared_kernel_times(torch, step, args.kernel_reps, max(3, args.kernel_iters // 2))
    step.run()
    torch.cuda.synchronize()
    snap = step.snapshot()
    for k in ref:
        if not torch.equal(ref[k], snap[k]):
            raise RuntimeError(f"benchmark output drifted in {k} ({w.spec.name})")
    rf, kernels, stages, shared, stage_us = rooflines(w, step.form, kern_us, shared_us)
    prog = progressive_timing(torch, w, dev)
    out = {"config": config_of(w, step.form, step.form == "two_streams", graph),
           "steps": steps, "ms_per_step": ms, "value": w.spec.B * w.spec.Nv / (ms * 1e-3),
           "unit": "visual tokens/s", "stream_choice_us": mode_us or None,
           "latency_us": {"kernels": kern_us, "kernels_shared_launches": shared_us or None,
                          "stages": stage_us},
           "roofline": rf, "roofline_kernels": kernels, "roofline_stages": stages,
           "roofline_kernels_shared_launches": shared or None, "progressive": prog,
           "csrc_digest": csrc_digest()}
    del graph, step
    torch.cuda.synchronize()
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cpu_baseline_one_sample(w)
    out["wall_s"] = round(time.perf_counter() - t0, 1)
    print(f"[bench] {w.spec.name}: {ms * 1000:.1f} us/step ({out['config']['step_form']}), "
          f"{out['wall_s']} s", file=sys.stderr, flush=True)
    return out


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
    if args.score_sweep:
        print(json.dumps(score_sweep(torch, dev)), flush=True)
        return
    if args.gemm_calibration:
        print(json.dumps(gemm_calibration(torch, dev)), flush=True)
        return
    w = W.make_workload(args.workload)
    s = w.spec
    step, ref, mode_us = prepare(w, dev, args)
    form = step.form
    split = form == "two_streams"

    if args.pmc_pass:
        # every dispatch of a library kernel here runs in the step's own
        # sequence (no graph, no back-to-back repeats)
        for _ in range(args.steps):
            step.run()
        torch.cuda.synchronize()
        n = args.calib_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty(n, dtype=torch.uint8, device=dev)
        src.fill_(1)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"pmc_pass": s.name, "step_form": form, "steps": args.steps,
                          "calib_bytes": n,
                          "csrc_digest": csrc_digest()}), flush=True)
        return

    # ---- headline: graph replay
    graph = None if args.no_graph else capture_step(torch, step, dev, ref)
    run_once = graph.replay if graph is not None else step.run
    ms_per_step = timed_steps(torch, run_once, args.steps, args.warmup)
    pct = replay_percentiles(torch, run_once)
    cold = cold_times(torch, step, dev, args.cold_mib) if args.cold_mib > 0 else None

    # ---- per-kernel durations (each kernel launched back to back between events)
    kern_us = kernel_times(torch, step, args.kernel_reps, args.kernel_iters)
    shared_us = shared_kernel_times(torch, step, args.kernel_reps, args.kernel_iters)
    breakdown = stage_breakdown(torch, step)

    for f in Step.FORMS:
        if f == form:
            continue

        def other(f=f):
            step.form = f
            try:
                step.run()
            finally:
                step.form = form
        breakdown["step_" + f] = graph_time_us(torch, other)
    vis_heads = visual_heads_timing(torch, step)
    crit_text = critical_text_timing(torch, step)
    prog = progressive_timing(torch, w, dev)
    step.run()
    torch.cuda.synchronize()
    # the outputs after all of the above still match the first eager step
    snap = step.snapshot()
    for k in ref:
        if not torch.equal(ref[k], snap[k]):
            raise RuntimeError(f"benchmark output drifted in {k}")
    rf, kernels, stages, shared, stage_us = rooflines(w, form, kern_us, shared_us)
    del graph, step
    torch.cuda.synchronize()

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
        "config": config_of(w, form, split, run_once if not args.no_graph else None),
        "latency_us": {"pipeline": ms_per_step * 1000.0, "pipeline_single_replays": pct,
                       "pipeline_cold": cold, "kernels": kern_us,
                       "kernels_shared_launches": shared_us or None,
                       "stages": stage_us, "calls_graph_replay": breakdown,
                       "stream_choice_us": mode_us or None},
        "roofline": rf,
        "roofline_kernels": kernels,
        "roofline_kernels_shared_launches": shared or None,
        "roofline_stages": stages,
        # outside the step: visual-head identification at the same layer and
        # critical text selection over the same text rows
        "visual_heads": vis_heads,
        "critical_text": crit_text,
        # the method's whole progressive schedule in one call
        "progressive": prog,
        "measured_peaks": measured_peaks(torch, dev),
        "csrc_digest": csrc_digest(),
    }
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    # the larger workloads: the same step and roofline figures, not the headline
    others = [int(x) for x in args.per_config.split(",") if x.strip()] if args.per_config else []
    per = {}
    for wid in others:
        if wid == args.workload:
            continue
        m = measure_other(torch, wid, dev, args)
        per[m["config"]["workload"]] = m
    if per:
        line["per_config"] = per
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
