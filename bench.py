#!/usr/bin/env python3
"""Stage-shard benchmark on one MI355X.

One step = forward + recompute + backward of one GPU's share of a GPT pipeline
stage for one micro-batch (every step of the hot path), run through the C ABI
of the HIP library: forward, recomputation and backward on two streams (the
library adds a third for the weight gradients).  Default workload: the 8.3B-shaped shard at
tensor-parallel degree 4 (6 blocks, hidden 3072, 32 heads / 8 local, FFN 12288
/ 3072 local, seq 1024, micro-batch 8 in 4 sub-micro-batches, recompute on 3
of 6 blocks, bf16).  Inputs are seeded synthetic tensors already resident in
HBM when timing starts.

Prints one JSON line (last line of stdout).

    python bench.py [--steps K] [--warmup W] [--config NAME] [--no-cpu-baseline]
                    [--n-sub N] [--mask M] [--streams 1|2] [--class-steps C]

`value` is executed FLOP per step over the mean step time of the K timed
steps (per-kernel timing off); the median and p10/p90 step times come from an
event per step boundary.  `roofline` is the kernel class with the largest
summed launch time per step, timed afterwards in a separate loop with HIP
events around every launch of one class at a time (on the stream each launch
runs on); `kernel_classes` lists every class.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2206_04959_amd import flops, synth  # noqa: E402

METRIC = "stage-shard fwd+bwd TFLOP/s per MI355X and % bf16 MFMA peak (8.3B-shaped, t=4)"
PEAK_BF16_TFLOPS = 2516.6   # dense bf16 MFMA: 256 CUs x 4096 FLOP/clk x 2.4 GHz
PEAK_HBM_GBS = 8000.0       # HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_gpt-8.3b-tp4.json")
CSRC = os.path.join(ROOT, "paper_2206_04959_amd", "csrc")


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def describe(s: synth.StageShape) -> str:
    return (f"{s.name} stage shard: {s.n_blocks} blocks, hidden {s.hidden}, {s.n_heads} heads "
            f"({s.local_heads} local, head_dim {s.head_dim}), ffn {s.ffn} ({s.local_ffn} local), seq {s.seq_len}, "
            f"micro-batch {s.micro_batch} in {s.n_sub} sub-micro-batches, tp_degree {s.tp_degree}, "
            f"recompute mask {bin(s.recompute_mask)}, {s.dtype}")


def sources_sha256() -> str:
    """One digest over every kernel source: counter data taken on other kernels is stale."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h", ".cpp")):
            h.update(name.encode())
            h.update(open(os.path.join(CSRC, name), "rb").read())
    return h.hexdigest()


def class_traffic(klass: str):
    """HBM bytes per launch of one kernel class, from the committed rocprofv3
    counter summary (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy of known
    size), or None if absent or taken on other kernel sources."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        if t.get("sources_sha256") != sources_sha256():
            return None
        return float(t["classes"][klass]["bytes_per_launch"])
    except (OSError, KeyError, ValueError, TypeError):
        return None


def class_rates(B, stage, step, shape, steps: int):
    """Per kernel class: HIP-event time of its launches over `steps` stage
    steps, and its algorithmic work per launch over that time against the
    roofline that bounds it."""
    import torch
    from paper_2206_04959_amd import kclass

    work = flops.class_work(shape)
    rows = []
    for name, (cid, desc) in kclass.CLASSES.items():
        stage.set_timing(cid)
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        ms, n = stage.read_timing()
        stage.set_timing(B.KC_NONE)
        amount, unit, bound = work[name]
        if n == 0:
            continue
        per_launch = amount * steps / n
        avg_ms = ms / n
        if unit == "FLOP":
            achieved, peak, u = per_launch / (avg_ms * 1e-3) / 1e12, PEAK_BF16_TFLOPS, "TFLOP/s"
        else:
            achieved, peak, u = per_launch / (avg_ms * 1e-3) / 1e9, PEAK_HBM_GBS, "GB/s"
        rows.append({"class": name, "kernel": desc, "bound": bound, "achieved": round(achieved, 2), "peak": peak,
                     "unit": u, "frac": round(achieved / peak, 4), "work_per_launch": per_launch,
                     "work_unit": unit, "launches_timed": n, "launches_per_step": n / steps,
                     "avg_launch_ms": round(avg_ms, 4), "launch_ms_per_step": round(ms / steps, 4)})
    total = sum(r["launch_ms_per_step"] for r in rows)
    for r in rows:
        r["share_of_launch_time"] = round(r["launch_ms_per_step"] / total, 4)
    return rows


def cpu_baseline(shape: synth.StageShape, budget_s: float = 15.0):
    """The fp64 oracle on a bounded sample of the same workload: one block of the
    shard, one sequence, forward + backward, repeated until about `budget_s`
    seconds of host time have been spent."""
    import numpy as np  # noqa: F401
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    sample = shape.replace(n_blocks=1, micro_batch=1, n_sub=1, recompute_mask=0, dtype="bf16")
    params = [{k: v.f64 for k, v in p.items()} for p in synth.stage_params(sample)]
    x = synth.stage_input(sample).f64
    dy = synth.upstream_grad(sample).f64
    reps, elapsed = 0, 0.0
    while reps == 0 or (elapsed < budget_s and reps < 200):
        t0 = time.perf_counter()
        oracle.shard_run(x, dy, params, sample.local_heads, sample.ln_eps)
        elapsed += time.perf_counter() - t0
        reps += 1
    work = flops.model_flops(sample) * reps
    return {"value": work / elapsed / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": (f"fp64 NumPy oracle, forward+backward of 1 block x 1 sequence of the {shape.name} shard "
                       f"({flops.model_flops(sample) / 1e9:.1f} GFLOP), {reps} run(s) in {elapsed:.1f} s")}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="gpt-8.3b-tp4", choices=sorted(synth.PRESETS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--class-steps", type=int, default=5, help="steps per kernel class in the launch-timing loop")
    ap.add_argument("--n-sub", type=int, default=None, help="sub-micro-batches per micro-batch (sweeps)")
    ap.add_argument("--mask", type=lambda v: int(v, 0), default=None, help="recompute mask (sweeps)")
    ap.add_argument("--streams", type=int, choices=(1, 2), default=2,
                    help="caller streams: 2 (sub-micro-batch j on stream j mod 2) or 1 (sweeps)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU's stage shard; --gpus {args.gpus} is not supported "
              "(the cross-GPU reductions are replaced by hand-off buffers on one GPU).", file=sys.stderr)
        return 2

    import torch
    from paper_2206_04959_amd import binding as B

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    shape = synth.PRESETS[args.config]
    if args.n_sub is not None:
        shape = shape.replace(n_sub=args.n_sub)
    if args.mask is not None:
        shape = shape.replace(recompute_mask=args.mask)
    log(f"[bench] {describe(shape)}")
    cfg = B.make_config(shape)
    params = B.to_device(B.pack_params(cfg, [{k: v.payload for k, v in p.items()}
                                              for p in synth.stage_params(shape)]))
    x = B.to_device(synth.stage_input(shape).payload)
    dy = B.to_device(synth.upstream_grad(shape).payload)
    y = torch.empty_like(x)
    dx = torch.empty_like(x)
    total, _ = B.param_layout(cfg)
    grads = torch.zeros(total, dtype=torch.float32, device="cuda")
    L, T, h = shape.n_blocks, shape.tokens, shape.hidden
    fwd_part = torch.empty((L, 2, T * h), dtype=x.dtype, device="cuda")
    bwd_part = torch.empty((L, 2, T * h), dtype=x.dtype, device="cuda")
    stage = B.Stage(shape)
    log(f"[bench] workspace {stage.workspace_bytes / 2**30:.2f} GiB, recompute area "
        f"{stage.recompute_bytes / 2**30:.2f} GiB")
    s0 = torch.cuda.Stream()
    s1 = torch.cuda.Stream() if args.streams == 2 else s0
    s0.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()

    def step():
        stage.fwd(params, x, y, fwd_part, streams=(s0, s1))
        # Recomputation on the backward's own streams, issued ahead of it.
        # Streams of its own, running beside the backward of the blocks that
        # kept their activations, measured slower: the step is throughput-
        # bound, and the extra co-running kernels cost more than they fill.
        stage.recompute(params, streams=(s0, s1))
        stage.bwd(params, dy, dx, grads, False, bwd_part, streams=(s0, s1))

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"[bench] warmup done ({args.warmup} steps)")

    # Headline: K steps with no per-kernel timing, one event per step boundary
    # on s0 (every call ends with s0 joined to the other streams).
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    marks[0].record(s0)
    for i in range(args.steps):
        step()
        marks[i + 1].record(s0)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    gpu_ms = marks[0].elapsed_time(marks[-1])
    per_step = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps))
    ms_per_step = gpu_ms / args.steps
    log(f"[bench] {args.steps} steps: {gpu_ms:.2f} ms on the GPU clock, {wall * 1e3:.2f} ms wall")

    # Per-class launch timing, in a separate loop after the headline: HIP
    # events around every launch of one kernel class at a time, on the stream
    # that launch runs on.
    classes = class_rates(B, stage, step, shape, args.class_steps)
    dominant = max(classes, key=lambda c: c["launch_ms_per_step"])
    traffic = class_traffic(dominant["class"])
    roof = {k: dominant[k] for k in ("bound", "achieved", "peak", "unit", "frac")}
    roof.update(traffic=traffic, kernel=dominant["kernel"], klass=dominant["class"],
                launches_timed=dominant["launches_timed"], launches_per_step=dominant["launches_per_step"],
                avg_launch_ms=dominant["avg_launch_ms"], work_per_launch=dominant["work_per_launch"],
                share_of_launch_time=dominant["share_of_launch_time"])

    exe = flops.executed_flops(shape)
    mdl = flops.model_flops(shape)
    value = exe / (ms_per_step * 1e-3) / 1e12

    def pct(q):
        return per_step[min(len(per_step) - 1, int(round(q * (len(per_step) - 1))))]

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if shape.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": describe(shape), "global_batch": shape.micro_batch, "seq_len": shape.seq_len,
                   "parallelism": f"tp{shape.tp_degree} shard on 1 GPU (cross-GPU reductions as hand-off buffers)"},
        "pct_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "step_ms_median": round(pct(0.5), 4),
        "step_ms_p10": round(pct(0.1), 4),
        "step_ms_p90": round(pct(0.9), 4),
        "tflops_at_median": round(exe / (pct(0.5) * 1e-3) / 1e12, 2),
        "executed_tflop_per_step": round(exe / 1e12, 4),
        "model_tflop_per_step": round(mdl / 1e12, 4),
        "model_tflops": round(mdl / (ms_per_step * 1e-3) / 1e12, 2),
        "streams": args.streams,
        "class_steps": args.class_steps,
        "workspace_bytes": stage.workspace_bytes,
        "recompute_area_bytes": stage.recompute_bytes,
        "roofline": roof,
        "kernel_classes": classes,
    }
    if not args.no_cpu_baseline:
        log("[bench] timing the oracle on the host (bounded sample)")
        out["cpu_baseline"] = cpu_baseline(shape)
    stage.close()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
