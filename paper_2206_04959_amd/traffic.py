"""HBM traffic of the grouped FC1/FC2 weight-gradient GEMM, from rocprofv3 counters.

Two steps, each run from the repository root on the GPU machine:

    rocprofv3 --pmc FETCH_SIZE -d <dir_f> -o run --output-format csv -- \
        python3 -m paper_2206_04959_amd.traffic run
    rocprofv3 --pmc WRITE_SIZE -d <dir_w> -o run --output-format csv -- \
        python3 -m paper_2206_04959_amd.traffic run
    python3 -m paper_2206_04959_amd.traffic summarize <dir_f> <dir_w>

`run` performs one fwd -> recompute -> bwd step of the 8.3B-shaped stage shard
(through the C ABI) and one plain copy kernel of a known size (an elementwise multiply by 1).
`summarize` reads both counter files, takes the counters of the grouped FC1/FC2
weight-gradient launches (the fp32-output GEMM with both operands read
transposed and the largest grid: the other weight-gradient launch of a block,
QKV and projection, has fewer tiles) and of the copy, scales the GEMM's readings by (known copy bytes / copy
reading), and writes profiles/gemm_dw_traffic.json, keyed by the SHA-256 of the
GEMM source so that a later kernel change invalidates it.
"""
from __future__ import annotations

import csv
import glob
import hashlib
import json
import os
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
OUT = os.path.join(ROOT, "profiles", "gemm_dw_traffic.json")
GEMM_SOURCE = os.path.join(PKG, "csrc", "gemm.hip")
COPY_BYTES = 512 * 2**20  # bytes read (and written) by the reference copy
DW_KERNEL = "true, true, 5>"  # template tail of the grouped dW GEMM instantiations (a_t, b_t, fp32 out)
COPY_KERNEL = "elementwise"   # torch's elementwise kernels (the reference copy is the last one run)


def run() -> None:
    sys.path.insert(0, ROOT)
    import torch
    from paper_2206_04959_amd import binding as B
    from paper_2206_04959_amd import synth

    shape = synth.PRESETS["gpt-8.3b-tp4"]
    cfg = B.make_config(shape)
    params = B.to_device(B.pack_params(cfg, [{k: v.payload for k, v in p.items()}
                                              for p in synth.stage_params(shape)]))
    x = B.to_device(synth.stage_input(shape).payload)
    dy = B.to_device(synth.upstream_grad(shape).payload)
    y, dx = torch.empty_like(x), torch.empty_like(x)
    total, _ = B.param_layout(cfg)
    grads = torch.zeros(total, dtype=torch.float32, device="cuda")
    stage = B.Stage(shape)
    s0, s1 = torch.cuda.Stream(), torch.cuda.Stream()
    s0.wait_stream(torch.cuda.current_stream())
    stage.fwd(params, x, y, streams=(s0, s1))
    stage.recompute(params, streams=(s0, s1))
    stage.bwd(params, dy, dx, grads, streams=(s0, s1))
    torch.cuda.synchronize()
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.mul(src, 1.0, out=dst)  # one elementwise kernel: reads and writes COPY_BYTES
    torch.cuda.synchronize()
    stage.close()
    print("traffic run done", flush=True)


def _dispatch_values(d: str, counter: str):
    """{dispatch id: (kernel name, grid size, summed counter value)} from one rocprofv3 output directory."""
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {d}")
    out = {}
    for f in files:
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            k = (f, int(r["Dispatch_Id"]))
            name, grid, v = out.get(k, (r["Kernel_Name"], int(r["Grid_Size"]), 0.0))
            out[k] = (name, grid, v + float(r["Counter_Value"]))
    return dict(sorted(out.items()))


def _pick(vals, needle: str, last_only: bool = False, largest_grid: bool = False):
    sel = [(grid, v) for (name, grid, v) in vals.values() if needle in name]
    if not sel:
        raise ValueError(f"no dispatch of a kernel containing {needle!r}")
    if largest_grid:
        g = max(grid for grid, _ in sel)
        sel = [(grid, v) for grid, v in sel if grid == g]
    sel = [v for _, v in sel]
    return sel[-1:] if last_only else sel


def summarize(dir_fetch: str, dir_write: str) -> dict:
    fetch = _dispatch_values(dir_fetch, "FETCH_SIZE")
    write = _dispatch_values(dir_write, "WRITE_SIZE")
    # counters are in KiB per dispatch
    f_copy = _pick(fetch, COPY_KERNEL, last_only=True)[0] * 1024.0
    w_copy = _pick(write, COPY_KERNEL, last_only=True)[0] * 1024.0
    f_scale, w_scale = COPY_BYTES / f_copy, COPY_BYTES / w_copy
    f_dw = [v * 1024.0 * f_scale for v in _pick(fetch, DW_KERNEL, largest_grid=True)]
    w_dw = [v * 1024.0 * w_scale for v in _pick(write, DW_KERNEL, largest_grid=True)]
    res = {
        "kernel": "grouped FC1/FC2 weight-gradient GEMM of one block (gpt-8.3b-tp4 stage shard)",
        "launches": len(f_dw),
        "fetch_bytes_per_launch": sum(f_dw) / len(f_dw),
        "write_bytes_per_launch": sum(w_dw) / len(w_dw),
        "copy_bytes": COPY_BYTES,
        "copy_fetch_reading_bytes": f_copy,
        "copy_write_reading_bytes": w_copy,
        "scale_fetch": f_scale,
        "scale_write": w_scale,
        "gemm_source_sha256": hashlib.sha256(open(GEMM_SOURCE, "rb").read()).hexdigest(),
        "commands": [
            "rocprofv3 --pmc FETCH_SIZE -d <dir_f> -o run --output-format csv -- "
            "python3 -m paper_2206_04959_amd.traffic run",
            "rocprofv3 --pmc WRITE_SIZE -d <dir_w> -o run --output-format csv -- "
            "python3 -m paper_2206_04959_amd.traffic run",
            "python3 -m paper_2206_04959_amd.traffic summarize <dir_f> <dir_w>",
        ],
    }
    res["bytes_per_launch"] = res["fetch_bytes_per_launch"] + res["write_bytes_per_launch"]
    os.makedirs(os.path.dirname(OUT), exist_ok=True)
    with open(OUT, "w") as f:
        json.dump(res, f, indent=1)
    return res


if __name__ == "__main__":
    if len(sys.argv) >= 2 and sys.argv[1] == "run":
        run()
    elif len(sys.argv) == 4 and sys.argv[1] == "summarize":
        print(json.dumps(summarize(sys.argv[2], sys.argv[3]), indent=1))
    else:
        print(__doc__)
        sys.exit(2)
