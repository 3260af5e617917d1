"""rocprofv3 counter summary of the isolated kernels (the kbench workload).

Three runs of the same command, then the summary (from the repository root on
the GPU machine):

    rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE --kernel-trace \
        -d <dir_m> -o run --output-format csv -- python3 -m paper_2206_04959_amd.kbench
    rocprofv3 --pmc FETCH_SIZE --kernel-trace -d <dir_f> -o run --output-format csv -- \
        python3 -m paper_2206_04959_amd.kbench
    rocprofv3 --pmc WRITE_SIZE --kernel-trace -d <dir_w> -o run --output-format csv -- \
        python3 -m paper_2206_04959_amd.kbench
    python3 -m paper_2206_04959_amd.counters <dir_m> <dir_f> <dir_w>

Per dispatch group (kernel name and grid size, in order of first appearance):
* GRBM_GUI_ACTIVE as rocprofv3 reports it is the sum over the 8 XCDs, so the
  GPU cycles of a dispatch are GRBM_GUI_ACTIVE / 8, and clock = that / kernel
  duration (the counting window is slightly longer than the kernel, so short
  kernels read high);
* SQ_VALU_MFMA_BUSY_CYCLES counts SIMD-cycles with the matrix core busy: for a
  GEMM it equals the ideal count, FLOP / 1024 per SIMD-cycle (dense bf16).
  MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GPU cycles x 256 CUs x 4 SIMDs), the
  matrix cores' utilisation at the clock the chip actually ran;
* HBM bytes = FETCH_SIZE and WRITE_SIZE (KiB per dispatch) scaled by what the
  same counters read for kbench's closing copy of known size, and the GB/s
  they give over the kernel's duration.
"""
from __future__ import annotations

import csv
import glob
import os
import sys
from collections import OrderedDict

COPY_BYTES = 512 * 2**20
N_CU, SIMD_PER_CU, N_XCD = 256, 4, 8


def _load(d: str):
    """{dispatch id: {name, grid, dur_ns, counters{}}} from one rocprofv3 run."""
    out = {}
    for f in glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            k = int(r["Dispatch_Id"])
            out.setdefault(k, {"name": r["Kernel_Name"], "grid": 0, "counters": {}})
            out[k]["dur_ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            k = int(r["Dispatch_Id"])
            e = out.setdefault(k, {"name": r["Kernel_Name"], "counters": {}})
            e["grid"] = int(r["Grid_Size"])
            c = e["counters"]
            c[r["Counter_Name"]] = c.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return dict(sorted(out.items()))


def _groups(disp):
    g = OrderedDict()
    for e in disp.values():
        if "dur_ns" not in e:
            continue
        g.setdefault((e["name"], e.get("grid", 0)), []).append(e)
    return g


def _short(name: str) -> str:
    if name.startswith("Cijk_"):
        return "hipBLASLt " + name.split("_MT")[1].split("_")[0] if "_MT" in name else "hipBLASLt"
    return name.replace("merak::", "").split("(")[0][:80]


def summarize(dir_m: str, dir_f: str, dir_w: str) -> str:
    gm = _groups(_load(dir_m))
    df, dw = _load(dir_f), _load(dir_w)

    def copy_reading(disp, counter):
        sel = [e["counters"].get(counter, 0.0) for e in disp.values() if "elementwise" in e["name"]]
        return sel[-1] * 1024.0

    f_scale = COPY_BYTES / copy_reading(df, "FETCH_SIZE")
    w_scale = COPY_BYTES / copy_reading(dw, "WRITE_SIZE")
    gf, gw = _groups(df), _groups(dw)
    lines = ["| kernel | grid | calls | avg us | clock GHz | MFMA busy | HBM read MB | HBM write MB | HBM GB/s |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for key, es in gm.items():
        name, grid = key
        if "merak" not in name and not name.startswith("Cijk_"):
            continue  # torch's input preparation and the calibration copy
        dur = sum(e["dur_ns"] for e in es) / len(es)
        grbm = sum(e["counters"].get("GRBM_GUI_ACTIVE", 0.0) for e in es) / len(es) / N_XCD
        busy = sum(e["counters"].get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) for e in es) / len(es)
        clk = grbm / dur if dur else 0.0
        util = busy / (grbm * N_CU * SIMD_PER_CU) if grbm else 0.0
        fe = gf.get(key, [])
        we = gw.get(key, [])
        rd = sum(e["counters"].get("FETCH_SIZE", 0.0) for e in fe) / max(len(fe), 1) * 1024.0 * f_scale
        wr = sum(e["counters"].get("WRITE_SIZE", 0.0) for e in we) / max(len(we), 1) * 1024.0 * w_scale
        gbs = (rd + wr) / dur if dur else 0.0
        lines.append(f"| `{_short(name)}` | {grid} | {len(es)} | {dur / 1e3:.1f} | {clk:.2f} | {util:.3f} | "
                     f"{rd / 1e6:.1f} | {wr / 1e6:.1f} | {gbs:.0f} |")
    lines.append(f"\nCopy calibration: FETCH_SIZE x {f_scale:.3f}, WRITE_SIZE x {w_scale:.3f} "
                 f"({COPY_BYTES >> 20} MiB copy).")
    return "\n".join(lines) + "\n"


if __name__ == "__main__":
    if len(sys.argv) != 4:
        print(__doc__)
        sys.exit(2)
    print(summarize(*sys.argv[1:]))
