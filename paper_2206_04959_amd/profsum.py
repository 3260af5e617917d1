"""Summary of a rocprofv3 kernel trace of bench.py, per kernel and per kernel class.

    rocprofv3 --kernel-trace --stats -d <dir> -o run --output-format csv -- \
        python3 -u bench.py --steps K --warmup W --no-cpu-baseline > <log>
    python3 -m paper_2206_04959_amd.profsum <dir> <log> "<the rocprofv3 command>"

Prints a markdown summary: every kernel instantiation's calls and durations,
every class's launches and kernel time per step (kclass.classify), and, for the
class the bench line reports as its roofline, the trace's average launch
duration next to the bench line's HIP-event figure.  The bench run times its
headline steps, then `class_steps` more steps per class (all visible in the
trace), so the trace's per-step figures divide by all steps the process ran.
"""
from __future__ import annotations

import csv
import glob
import json
import os
import sys
from collections import defaultdict


def _rows(d: str):
    files = glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no kernel_trace.csv under {d}")
    for f in files:
        yield from csv.DictReader(open(f))


def summarize(d: str, log: str, command: str) -> str:
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from paper_2206_04959_amd import kclass

    line = None
    for l in open(log):
        l = l.strip()
        if l.startswith("{") and '"metric"' in l:
            line = json.loads(l)
    if line is None:
        raise ValueError(f"no bench line in {log}")
    n_steps = line["warmup"] + line["steps"] + len(line["kernel_classes"]) * line.get("class_steps", 5)
    rows = [r for r in _rows(d)]
    durs = defaultdict(list)
    grids = {}
    for r in rows:
        name = r["Kernel_Name"]
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        durs[name].append(us)
        grids.setdefault(name, []).append(int(r.get("Grid_Size", r.get("Grid_Size_X", 0)) or 0))
    dw_grids = tuple(sorted({g for n, gs in grids.items() if kclass.is_dw(n) for g in gs}))
    per_class = defaultdict(list)
    for r in rows:
        name = r["Kernel_Name"]
        grid = int(r.get("Grid_Size", r.get("Grid_Size_X", 0)) or 0)
        c = kclass.classify(name, grid, dw_grids)
        if c:
            per_class[c].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    total_us = sum(sum(v) for v in durs.values())
    out = []
    out.append("Command (run from the repository root on the GPU machine):\n")
    out.append("```\n" + command + "\n```\n")
    out.append(f"Bench line of the profiled run: {line['value']} TFLOP/s, {line['ms_per_step']} ms per step "
               f"(median {line.get('step_ms_median')}, p10 {line.get('step_ms_p10')}, p90 {line.get('step_ms_p90')}).\n")
    out.append(f"Stage steps run by the process (warm-up, timed, class-timing loop): {n_steps}. "
               f"Kernel time summed over all streams: {total_us / 1e3:.2f} ms "
               f"({total_us / 1e3 / n_steps:.2f} ms per step; the streams overlap, so this exceeds the wall time).\n")
    out.append("## Kernels\n")
    out.append("| kernel | calls | per step ms | avg us | min us | max us | share |")
    out.append("|---|---:|---:|---:|---:|---:|---:|")
    for name, v in sorted(durs.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"| `{name[:110]}` | {len(v)} | {sum(v) / 1e3 / n_steps:.3f} | {sum(v) / len(v):.1f} | "
                   f"{min(v):.1f} | {max(v):.1f} | {100 * sum(v) / total_us:.1f}% |")
    out.append("\n## Kernel classes\n")
    out.append("| class | launches per step | kernel ms per step | avg launch us (trace) | "
               "avg launch us (bench events) |")
    out.append("|---|---:|---:|---:|---:|")
    ev = {c["class"]: c for c in line["kernel_classes"]}
    for c, v in sorted(per_class.items(), key=lambda kv: -sum(kv[1])):
        # the attention backward is one launch of the timing class but two kernels
        pair = 2 if c == "ATTN_BWD" else 1
        trace_avg = sum(v) / (len(v) / pair)
        e = ev.get(c)
        out.append(f"| {c} | {len(v) / pair / n_steps:.1f} | {sum(v) / 1e3 / n_steps:.3f} | {trace_avg:.1f} | "
                   f"{e['avg_launch_ms'] * 1e3:.1f} |" if e else
                   f"| {c} | {len(v) / pair / n_steps:.1f} | {sum(v) / 1e3 / n_steps:.3f} | {trace_avg:.1f} | - |")
    roof = line["roofline"]
    rc = roof.get("klass")
    if rc in per_class:
        v = per_class[rc]
        pair = 2 if rc == "ATTN_BWD" else 1
        trace_avg = sum(v) / (len(v) / pair)
        out.append(f"\nRoofline class of the bench line: {rc}. Bench (HIP events on the launching stream): "
                   f"{roof['avg_launch_ms'] * 1e3:.1f} us per launch, {roof['achieved']} {roof['unit']} "
                   f"(frac {roof['frac']}). Trace (first to last wave): {trace_avg:.1f} us per launch, "
                   f"{roof['work_per_launch'] / (trace_avg * 1e-6) / 1e12:.1f} TFLOP/s "
                   f"(frac {roof['work_per_launch'] / (trace_avg * 1e-6) / 1e12 / roof['peak']:.4f}). "
                   "An event interval also covers the wait for CUs held by the other streams, so it is the "
                   "longer of the two.")
    return "\n".join(out) + "\n"


if __name__ == "__main__":
    if len(sys.argv) != 4:
        print(__doc__)
        sys.exit(2)
    print(summarize(sys.argv[1], sys.argv[2], sys.argv[3]))
