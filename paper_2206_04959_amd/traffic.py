"""HBM traffic of every kernel class of the stage step, from rocprofv3 counters.

Two steps, each run from the repository root on the GPU machine:

    rocprofv3 --pmc FETCH_SIZE -d <dir_f> -o run --output-format csv -- \
        python3 -m paper_2206_04959_amd.traffic run
    rocprofv3 --pmc WRITE_SIZE -d <dir_w> -o run --output-format csv -- \
        python3 -m paper_2206_04959_amd.traffic run
    python3 -m paper_2206_04959_amd.traffic summarize <dir_f> <dir_w>

`run` performs one fwd -> recompute -> bwd step of the 8.3B-shaped stage shard
(through the C ABI) and one plain copy kernel of a known size (an elementwise
multiply by 1).  `summarize` reads both counter files, assigns every dispatch
of the step to its kernel class (kclass.classify), scales the readings by
(known copy bytes / the copy's reading) and writes
profiles/traffic_gpt-8.3b-tp4.json: per class the launches of one step and the
fetched and written bytes per launch, keyed by a digest of the kernel sources
so that a later kernel change invalidates it.
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
OUT = os.path.join(ROOT, "profiles", "traffic_gpt-8.3b-tp4.json")
CSRC = os.path.join(PKG, "csrc")
COPY_BYTES = 512 * 2**20  # bytes read (and written) by the reference copy
COPY_KERNEL = "elementwise"   # torch's elementwise kernels (the reference copy is the last one run)


def sources_sha256() -> str:
    """One digest over every kernel source (the same one bench.py checks)."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h", ".cpp")):
            h.update(name.encode())
            h.update(open(os.path.join(CSRC, name), "rb").read())
    return h.hexdigest()


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


def _copy_reading(vals) -> float:
    sel = [v for (name, grid, v) in vals.values() if COPY_KERNEL in name]
    if not sel:
        raise ValueError("no dispatch of the reference copy")
    return sel[-1] * 1024.0  # counters are in KiB per dispatch


def _per_class(vals, scale: float):
    sys.path.insert(0, ROOT)
    from paper_2206_04959_amd import kclass
    dw_grids = tuple(sorted({grid for (name, grid, v) in vals.values() if kclass.is_dw(name)}))
    out = {}
    for name, grid, v in vals.values():
        c = kclass.classify(name, grid, dw_grids)
        if c is None:
            continue
        n, tot = out.get(c, (0, 0.0))
        out[c] = (n + 1, tot + v * 1024.0 * scale)
    return out


def summarize(dir_fetch: str, dir_write: str) -> dict:
    fetch = _dispatch_values(dir_fetch, "FETCH_SIZE")
    write = _dispatch_values(dir_write, "WRITE_SIZE")
    f_copy, w_copy = _copy_reading(fetch), _copy_reading(write)
    f_scale, w_scale = COPY_BYTES / f_copy, COPY_BYTES / w_copy
    fc, wc = _per_class(fetch, f_scale), _per_class(write, w_scale)
    classes = {}
    for c in sorted(set(fc) | set(wc)):
        nf, bf = fc.get(c, (0, 0.0))
        nw, bw = wc.get(c, (0, 0.0))
        n = max(nf, nw, 1)
        classes[c] = {"launches": n, "fetch_bytes_per_launch": bf / max(nf, 1),
                      "write_bytes_per_launch": bw / max(nw, 1),
                      "bytes_per_launch": bf / max(nf, 1) + bw / max(nw, 1)}
    res = {
        "workload": "gpt-8.3b-tp4 stage shard, one fwd -> recompute -> bwd step",
        "classes": classes,
        "copy_bytes": COPY_BYTES,
        "copy_fetch_reading_bytes": f_copy,
        "copy_write_reading_bytes": w_copy,
        "scale_fetch": f_scale,
        "scale_write": w_scale,
        "sources_sha256": sources_sha256(),
        "commands": [
            "rocprofv3 --pmc FETCH_SIZE -d <dir_f> -o run --output-format csv -- "
            "python3 -m paper_2206_04959_amd.traffic run",
            "rocprofv3 --pmc WRITE_SIZE -d <dir_w> -o run --output-format csv -- "
            "python3 -m paper_2206_04959_amd.traffic run",
            "python3 -m paper_2206_04959_amd.traffic summarize <dir_f> <dir_w>",
        ],
    }
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
