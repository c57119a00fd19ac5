"""Turns rocprofv3 output of bench.py runs into the short text summaries kept
with the sources.

  python -m paper_2608_25332_amd.profile_summary trace <kernel_stats.csv> \\
      --workload NAME --command "CMD"                      > summary.md
  python -m paper_2608_25332_amd.profile_summary pmc <fetch counter_collection.csv> \\
      <write counter_collection.csv> --workload NAME --calib-bytes N \\
      --digest D --command "CMD" --command2 "CMD2"        > summary.md
  python -m paper_2608_25332_amd.profile_summary counters <counter_collection.csv>... \\
      --workload NAME --command "CMD" [--command "CMD2"] --note TEXT > summary.md

pmc: FETCH_SIZE and WRITE_SIZE (KiB per dispatch, summed over the L2
channels) of every library kernel, averaged over its dispatches and scaled
by what the same counter reads for the calibration copy (a plain copy kernel
of calib-bytes read and written), so that the figures are in bytes of HBM
traffic.  The JSON block at the end is what bench.py reads; `csrc_digest`
ties the figures to the library sources they were taken from.
"""

from __future__ import annotations

import argparse
import csv
import json
import sys
from collections import defaultdict


def short(name: str) -> str:
    n = name.split("(")[0].replace("void ", "")
    if n.startswith("pv::"):
        n = n[4:]
    return n


def kernel_key(name: str) -> str:
    """Library kernel name without template arguments (cos_partial, ...)."""
    n = short(name).split("<")[0]
    return n[:-len("_kernel")] if n.endswith("_kernel") else n


def split_trace(path: str):
    """Per kernel: mean duration (us) of the dispatches that ran in runs of at
    least 10 identical back-to-back launches (what bench.py times with HIP
    events) and of the others (the step's own sequence)."""
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    names = [short(r["Kernel_Name"]) for r in rows]
    grid = [(r["Grid_Size_X"], r.get("Grid_Size_Y", "1"), r.get("Grid_Size_Z", "1")) for r in rows]
    dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rows]
    b2b, seq = defaultdict(list), defaultdict(list)
    i = 0
    while i < len(rows):
        j = i
        while j + 1 < len(rows) and names[j + 1] == names[i] and grid[j + 1] == grid[i]:
            j += 1
        (b2b if j - i + 1 >= 10 else seq)[names[i]].extend(dur[i:j + 1])
        i = j + 1
    mean = lambda v: sum(v) / len(v) if v else float("nan")
    return {n: (mean(b2b[n]), mean(seq[n])) for n in set(b2b) | set(seq)}


def b2b_by_shape(path: str):
    """Mean duration (us) and count of the back-to-back dispatches (runs of at
    least 10 identical launches) per (kernel, grid size in work-items)."""
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    key = [(short(r["Kernel_Name"]), "x".join(r.get(f"Grid_Size_{a}", "1") for a in "XYZ"))
           for r in rows]
    dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rows]
    out = defaultdict(list)
    i = 0
    while i < len(rows):
        j = i
        while j + 1 < len(rows) and key[j + 1] == key[i]:
            j += 1
        if j - i + 1 >= 10:
            out[key[i]].extend(dur[i:j + 1])
        i = j + 1
    return {k: (sum(v) / len(v), len(v)) for k, v in out.items()}


def trace(args) -> str:
    rows = list(csv.DictReader(open(args.stats)))
    split = split_trace(args.trace_csv) if args.trace_csv else {}
    bench = json.load(open(args.bench_json)) if args.bench_json else None
    out = [f"# Kernel trace: {args.workload}", "",
           "Command (repository root on one MI355X; rocprofv3 writes under gpurun_out/):", "",
           "```", args.command, "```", "",
           "rocprofv3 `--kernel-trace --stats`, library kernels.  `avg` is over every dispatch of",
           "the run; `back-to-back` over the dispatches bench.py times with HIP events (each",
           "kernel launched repeatedly); `in step` over the dispatches inside the step's own",
           "sequence (graph replays: the previous kernel was a different one).", "",
           "| kernel | calls | avg us | back-to-back us | in step us | min us | max us |",
           "|---|---|---|---|---|---|---|"]
    for r in rows:
        if not r["Name"].startswith(("pv::", "void pv::")):
            continue
        n = short(r["Name"])
        b, q = split.get(n, (float("nan"), float("nan")))
        out.append(f"| `{n}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | {b:.2f} | "
                   f"{q:.2f} | {float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} |")
    if args.trace_csv:
        shapes = b2b_by_shape(args.trace_csv)
        out += ["", "Back-to-back dispatches by launch shape (grid in work-items; the kernels "
                "that carry another step's workgroups run at their own shapes):", "",
                "| kernel | grid | dispatches | avg us |", "|---|---|---|---|"]
        for (n, g), (us, cnt) in sorted(shapes.items()):
            if n.startswith("pv::") or "_kernel" in n:
                out.append(f"| `{n}` | {g} | {cnt} | {us:.2f} |")
    if bench:
        ks = bench["latency_us"]["kernels"]
        rf = bench["roofline"]
        out += ["", "The same run's bench.py line, HIP-event average per launch (us), the four "
                "calls made separately:", "", "| kernel | us |", "|---|---|"]
        out += [f"| {k} | {v:.2f} |" for k, v in ks.items()]
        sh = bench["latency_us"].get("kernels_shared_launches")
        if sh:
            out += ["", "and the launches of the one-call step (pv_prune_pipeline_timed):", "",
                    "| kernel | us |", "|---|---|"]
            out += [f"| {k} | {v:.2f} |" for k, v in sh.items()]
        out += ["", f"Step (HIP-graph replay): {bench['latency_us']['pipeline']:.2f} us, "
                f"{bench['value'] / 1e6:.2f} M visual tokens/s.  Dominant kernel "
                f"`{rf['kernel']}`: {rf['kernel_us']:.2f} us by HIP events."]
    return "\n".join(out) + "\n"


def counter_values(path: str, counter: str):
    """Counter value of every dispatch (summed over dimensions), per kernel."""
    per_dispatch = defaultdict(float)
    names = {}
    for r in csv.DictReader(open(path)):
        if r.get("Counter_Name") != counter:
            continue
        key = r["Dispatch_Id"]
        per_dispatch[key] += float(r["Counter_Value"])
        names[key] = r["Kernel_Name"]
    acc = defaultdict(list)
    for key, v in per_dispatch.items():
        acc[names[key]].append(v)
    return acc


def calib_kib(values) -> float:
    """Counter KiB of the calibration copy: the mean over the copy-kernel
    dispatches within half of the largest one (the large copies; the
    runtime's small copies use the same kernel)."""
    big = [v for n, vs in values.items() if "copyBuffer" in n for v in vs]
    if not big:
        sys.exit("no calibration copy kernel in the run")
    top = max(big)
    sel = [v for v in big if v >= 0.5 * top]
    return sum(sel) / len(sel)


def pmc(args) -> str:
    fetch = counter_values(args.fetch, "FETCH_SIZE")
    write = counter_values(args.write, "WRITE_SIZE")
    kib = 1024.0
    cf, cw = calib_kib(fetch), calib_kib(write)
    f_scale = args.calib_bytes / (cf * kib)
    w_scale = args.calib_bytes / (cw * kib)
    mean = lambda v: sum(v) / len(v)
    kern = {}
    for n, fv in fetch.items():
        if not n.startswith(("pv::", "void pv::")):
            continue
        k = kernel_key(n)
        wv = mean(write[n]) if n in write else 0.0
        kern[k] = {"fetch_bytes": mean(fv) * kib * f_scale, "write_bytes": wv * kib * w_scale,
                   "dispatches": len(fv), "fetch_kib_raw": mean(fv), "write_kib_raw": wv}
    out = [f"# HBM traffic per dispatch: {args.workload}", "",
           "Commands (repository root on one MI355X, one counter per run):", "",
           "```", args.command, args.command2, "```", "",
           f"Calibration: a {args.calib_bytes} B device copy (the runtime's copy kernel) "
           f"reads {cf:.0f} KiB (FETCH_SIZE) and writes {cw:.0f} KiB (WRITE_SIZE); "
           f"scale factors {f_scale:.4f} (fetch) and {w_scale:.4f} (write) turn counter KiB "
           "into bytes.", "",
           "| kernel | dispatches | fetch KiB (raw) | write KiB (raw) | fetch bytes | write bytes |",
           "|---|---|---|---|---|---|"]
    for k, v in sorted(kern.items()):
        out.append(f"| {k} | {v['dispatches']} | {v['fetch_kib_raw']:.1f} | "
                   f"{v['write_kib_raw']:.1f} | {v['fetch_bytes']:.0f} | {v['write_bytes']:.0f} |")
    rec = {"workload": args.workload, "csrc_digest": args.digest,
           "kernels": {k: {"fetch_bytes": round(v["fetch_bytes"]), "write_bytes":
                           round(v["write_bytes"])} for k, v in kern.items()}}
    out += ["", "```json", json.dumps(rec, indent=1), "```"]
    return "\n".join(out) + "\n"


def counters(args) -> str:
    """Per library kernel, the mean per dispatch of every counter in the given
    counter_collection.csv files (one rocprofv3 --pmc run each)."""
    vals = defaultdict(lambda: defaultdict(list))
    for path in args.csv:
        rows = list(csv.DictReader(open(path)))
        per = defaultdict(float)
        names = {}
        for r in rows:
            key = (r["Dispatch_Id"], r["Counter_Name"])
            per[key] += float(r["Counter_Value"])
            names[r["Dispatch_Id"]] = r["Kernel_Name"]
        for (disp, cname), v in per.items():
            n = names[disp]
            if n.startswith(("pv::", "void pv::")):
                vals[kernel_key(n)][cname].append(v)
    cnames = sorted({c for d in vals.values() for c in d})
    out = [f"# Hardware counters per dispatch: {args.workload}", "",
           "Commands (repository root on one MI355X, one run per line):", "", "```"]
    out += list(args.command) + ["```", "", args.note, "",
                                 "| kernel | dispatches | " + " | ".join(cnames) + " |",
                                 "|---|---|" + "---|" * len(cnames)]
    for k, d in sorted(vals.items()):
        n = max(len(v) for v in d.values())
        cells = []
        for c in cnames:
            v = d.get(c)
            cells.append("" if not v else f"{sum(v) / len(v):.1f}")
        out.append(f"| {k} | {n} | " + " | ".join(cells) + " |")
    return "\n".join(out) + "\n"


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("trace")
    t.add_argument("stats")
    t.add_argument("--workload", required=True)
    t.add_argument("--command", required=True)
    t.add_argument("--trace-csv", help="kernel_trace.csv of the same run")
    t.add_argument("--bench-json", help="bench.py's JSON line from the same run")
    p = sub.add_parser("pmc")
    p.add_argument("fetch")
    p.add_argument("write")
    p.add_argument("--workload", required=True)
    p.add_argument("--calib-bytes", type=int, required=True)
    p.add_argument("--digest", required=True)
    p.add_argument("--command", required=True)
    p.add_argument("--command2", required=True)
    c = sub.add_parser("counters")
    c.add_argument("csv", nargs="+")
    c.add_argument("--workload", required=True)
    c.add_argument("--command", action="append", required=True)
    c.add_argument("--note", default="")
    a = ap.parse_args(argv)
    sys.stdout.write({"trace": trace, "pmc": pmc, "counters": counters}[a.cmd](a))


if __name__ == "__main__":
    main()
