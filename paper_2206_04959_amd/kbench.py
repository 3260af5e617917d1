"""Isolated rate of every kernel class of the stage, at the shapes one launch
of the gpt-8.3b-tp4 stage shard uses, each against the roofline that bounds it.

    python3 -m paper_2206_04959_amd.kbench

One stream, one kernel at a time, random bf16 inputs resident in HBM, HIP
events around `iters` back-to-back calls through the C ABI.  Inside the stage
step these kernels share the GPU with one to two others, so their in-step
durations (the kernel trace) are longer; this table is what each kernel does
with the whole chip.

Shapes: a stream's grouped launch covers two sub-micro-batches (4096 token
rows); the weight-gradient GEMMs reduce over the whole micro-batch (K = 8192).
GEMM FLOP = 2 M N K.  Attention FLOP = 2 B H d S (S + 1) forward (causal:
Q K^T and P V over the lower triangle including the diagonal) and twice that
backward (dV, dP, dQ, dK over the same pairs; P rebuilt from lse is not
counted).  Every GEMM also runs through torch.matmul (hipBLASLt) on the same
shape as a yardstick (plain product, no epilogue).  Memory-
bound kernels count the bytes they must move once: LayerNorm forward reads x
and writes y (2 rows of h bf16 values per row), the backward reads dout, x and
the residual gradient and writes dx (its parameter sums re-read dout and x,
which is not counted); the column sum reads its input once.
Peaks: dense bf16 MFMA 2516.6 TFLOP/s, HBM 8 TB/s.
"""
from __future__ import annotations

import os
import sys

PEAK_TF = 2516.6
PEAK_GBS = 8000.0


def main() -> None:
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import torch

    from paper_2206_04959_amd import binding as B

    if not torch.cuda.is_available():
        raise SystemExit("kbench needs a GPU")
    torch.manual_seed(0)
    dev = "cuda"
    iters = int(os.environ.get("KBENCH_ITERS", "30"))
    h, hl, fl, T, Ms = 3072, 768, 3072, 8192, 4096

    def bf(*shape, std=0.5):
        return (torch.randn(*shape, device=dev) * std).to(torch.bfloat16)

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters * 1e3  # us

    rows = []

    def gemm_row(name, M, N, K, a_t, b_t, epi):
        a = bf(K, M) if a_t else bf(M, K)
        b = bf(K, N) if b_t else bf(N, K)
        c = torch.empty((M, N), device=dev, dtype=torch.float32 if epi == B.EPI_F32 else torch.bfloat16)
        bias, aux, resid = bf(N, std=0.1), bf(M, N), bf(M, N)
        us = timed(lambda: B.gemm(a, b, c, M, N, K, a_trans=a_t, b_trans=b_t, epilogue=epi, bias=bias,
                                  resid=resid, aux=aux))
        tf = 2.0 * M * N * K / us / 1e6
        A = a.t() if a_t else a
        Bm = b if b_t else b.t()
        ref_us = timed(lambda: torch.matmul(A, Bm))
        rows.append((name, f"{M}x{N}x{K}", us, f"{tf:.0f} TFLOP/s", tf / PEAK_TF, "mfma",
                     f"{2.0 * M * N * K / ref_us / 1e6:.0f} TFLOP/s ({ref_us:.1f} us)"))

    gemm_row("QKV forward (bias)", Ms, 3 * hl, h, False, False, B.EPI_BIAS)
    gemm_row("projection forward (bias + residual + hand-off)", Ms, h, hl, False, False, B.EPI_BIAS_RESID)
    gemm_row("FC1 forward (bias + GeLU, keeps u)", Ms, fl, h, False, False, B.EPI_BIAS_GELU)
    gemm_row("FC2 forward (bias + residual + hand-off)", Ms, h, fl, False, False, B.EPI_BIAS_RESID)
    gemm_row("FC2 input gradient (x GeLU')", Ms, fl, h, False, True, B.EPI_GELU_BWD)
    gemm_row("FC1 input gradient", Ms, h, fl, False, True, B.EPI_STORE)
    gemm_row("projection input gradient", Ms, hl, h, False, True, B.EPI_STORE)
    gemm_row("QKV input gradient", Ms, h, 3 * hl, False, True, B.EPI_STORE)
    gemm_row("FC2 weight gradient (one of the grouped pair)", h, fl, T, True, True, B.EPI_F32)

    bt, S, H, D = 4, 1024, 8, 96
    qkv = bf(bt, S, 3, H, D)
    o = torch.empty(bt, S, H, D, device=dev, dtype=torch.bfloat16)
    lse = torch.empty(bt, H, S, device=dev, dtype=torch.float32)
    do = bf(bt, S, H, D)
    dqkv = torch.empty_like(qkv)
    delta = torch.empty(bt, H, S, device=dev, dtype=torch.float32)
    fl_att = 2.0 * bt * H * D * S * (S + 1)
    us = timed(lambda: B.attention_fwd(qkv, o, lse, bt, S, H, D))
    rows.append(("attention forward", f"{bt}x{S} seq, {H} heads, d {D}", us, f"{fl_att / us / 1e6:.0f} TFLOP/s",
                 fl_att / us / 1e6 / PEAK_TF, "mfma"))
    us = timed(lambda: B.attention_bwd(qkv, o, lse, do, dqkv, delta, bt, S, H, D))
    rows.append(("attention backward (dQ with delta, dK/dV)", f"{bt}x{S} seq, {H} heads, d {D}", us,
                 f"{2.0 * fl_att / us / 1e6:.0f} TFLOP/s", 2.0 * fl_att / us / 1e6 / PEAK_TF, "mfma"))

    x, g, be = bf(Ms, h, std=2.0), bf(h, std=0.1), bf(h, std=0.1)
    y = torch.empty_like(x)
    mean = torch.empty(Ms, device=dev, dtype=torch.float32)
    rstd = torch.empty(Ms, device=dev, dtype=torch.float32)
    us = timed(lambda: B.layernorm_fwd(x, g, be, y, mean, rstd))
    gbs = 2.0 * Ms * h * 2 / us / 1e3
    rows.append(("LayerNorm forward", f"{Ms}x{h}", us, f"{gbs:.0f} GB/s", gbs / PEAK_GBS, "hbm"))
    dout, dres = bf(Ms, h), bf(Ms, h)
    dxl = torch.empty_like(x)
    dg = torch.empty(h, device=dev, dtype=torch.float32)
    db = torch.empty(h, device=dev, dtype=torch.float32)
    scratch = torch.empty(2 * B.reduce_scratch_elems(Ms, h), device=dev, dtype=torch.float32)
    us = timed(lambda: B.layernorm_bwd(dout, x, mean, rstd, g, dres, dxl, dg, db, scratch))
    gbs = 4.0 * Ms * h * 2 / us / 1e3
    rows.append(("LayerNorm backward with parameter sums", f"{Ms}x{h}", us, f"{gbs:.0f} GB/s", gbs / PEAK_GBS,
                 "hbm"))
    xs = bf(T, h)
    out = torch.empty(h, device=dev, dtype=torch.float32)
    cs = torch.empty(B.reduce_scratch_elems(T, h), device=dev, dtype=torch.float32)
    us = timed(lambda: B.column_sum(xs, out, cs))
    gbs = 1.0 * T * h * 2 / us / 1e3
    rows.append(("bias gradient (column sum)", f"{T}x{h}", us, f"{gbs:.0f} GB/s", gbs / PEAK_GBS, "hbm"))

    # a plain copy of known size last (counter calibration for the HBM byte counts)
    src = torch.empty(512 * 2**20 // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()

    print("| kernel | shape | us | rate | fraction of peak | bound | hipBLASLt, same shape |")
    print("|---|---|---:|---:|---:|---|---:|")
    for r in rows:
        name, shape, us, rate, frac, bound = r[:6]
        ref = r[6] if len(r) > 6 else "-"
        print(f"| {name} | {shape} | {us:.1f} | {rate} | {frac:.3f} | {bound} | {ref} |")


if __name__ == "__main__":
    main()
