"""Per-kernel parity of the HIP kernels (through the C ABI's per-kernel entry
points) against the oracle's building blocks / the plain definition."""
import numpy as np
import pytest

import oracle
from paper_2206_04959_amd import binding as B
from paper_2206_04959_amd import synth
from tests.gpu_util import need_gpu, rel_err

pytestmark = pytest.mark.gpu


def _rand(shape, dtype, seed, std=1.0, mean=0.0):
    rng = np.random.default_rng(seed)
    v = (rng.standard_normal(size=shape, dtype=np.float32) * np.float32(std) + np.float32(mean))
    if dtype == "bf16":
        bits = synth.f32_to_bf16_bits(v)
        return bits, synth.bf16_bits_to_f64(bits)
    return v, v.astype(np.float64)


def _dev(payload):
    return B.to_device(payload)


GEMM_SHAPES = [(192, 320, 128), (2048, 8192, 128), (320, 192, 512)]


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("a_t,b_t", [(0, 0), (0, 1), (1, 1), (1, 0)])
@pytest.mark.parametrize("mnk", GEMM_SHAPES)
def test_gemm_layouts(dtype, a_t, b_t, mnk):
    torch = need_gpu()
    M, N, K = mnk
    if dtype == "fp32" and M * N > 4_000_000:
        pytest.skip("large fp32 case not needed")
    print(f"[gemm] {dtype} a_t={a_t} b_t={b_t} {mnk}", flush=True)
    a_p, a = _rand((K, M) if a_t else (M, K), dtype, 1)
    b_p, b = _rand((K, N) if b_t else (N, K), dtype, 2)
    A = a.T if a_t else a
    Bm = b if b_t else b.T
    ref = A @ Bm
    c = torch.empty((M, N), dtype=torch.bfloat16 if dtype == "bf16" else torch.float32, device="cuda")
    B.gemm(_dev(a_p), _dev(b_p), c, M, N, K, a_trans=a_t, b_trans=b_t, epilogue=B.EPI_STORE)
    torch.cuda.synchronize()
    tol = 1e-2 if dtype == "bf16" else 1e-5
    assert rel_err(B.to_host_f64(c), ref) < tol
    # fp32 output (the weight-gradient epilogue), overwrite then accumulate
    c32 = torch.empty((M, N), dtype=torch.float32, device="cuda")
    B.gemm(_dev(a_p), _dev(b_p), c32, M, N, K, a_trans=a_t, b_trans=b_t, epilogue=B.EPI_F32,
           dtype=B.BF16 if dtype == "bf16" else B.FP32)
    B.gemm(_dev(a_p), _dev(b_p), c32, M, N, K, a_trans=a_t, b_trans=b_t, epilogue=B.EPI_F32, accumulate=True,
           dtype=B.BF16 if dtype == "bf16" else B.FP32)
    torch.cuda.synchronize()
    assert rel_err(c32.cpu().numpy(), 2 * ref) < 2e-5


@pytest.mark.parametrize("cfg", list(range(1, 11)))
@pytest.mark.parametrize("a_t,b_t", [(0, 0), (0, 1), (1, 1), (1, 0)])
def test_gemm_smallest_problem_on_every_tile(cfg, a_t, b_t):
    """M = N = K = 64, the smallest problem the boundary accepts: one partial
    tile of every shape (up to 256 x 256), one K stage."""
    torch = need_gpu()
    M = N = K = 64
    print(f"[gemm 64^3] tile {cfg} a_t={a_t} b_t={b_t}", flush=True)
    a_p, a = _rand((K, M) if a_t else (M, K), "bf16", 23)
    b_p, b = _rand((K, N) if b_t else (N, K), "bf16", 24)
    ref = (a.T if a_t else a) @ (b if b_t else b.T)
    c32 = torch.empty((M, N), dtype=torch.float32, device="cuda")
    prev = B.gemm_tile_override(cfg)
    try:
        B.gemm(_dev(a_p), _dev(b_p), c32, M, N, K, a_trans=a_t, b_trans=b_t, epilogue=B.EPI_F32, dtype=B.BF16)
        torch.cuda.synchronize()
    finally:
        B.gemm_tile_override(prev)
    assert rel_err(c32.cpu().numpy(), ref) < 2e-5


# bf16: the automatic tile choice and each tile the stage's choice can make
# (256x256, 256x128 and 128x192 tiles, 256x192); fp32 has one kernel.
EPI_CASES = [("bf16", 0), ("bf16", 7), ("bf16", 8), ("bf16", 9), ("bf16", 10), ("fp32", 0)]


@pytest.mark.parametrize("dtype,tile", EPI_CASES)
def test_gemm_epilogues(dtype, tile):
    torch = need_gpu()
    print(f"[gemm epilogues] {dtype} tile {tile}", flush=True)
    prev = B.gemm_tile_override(tile)
    try:
        _gemm_epilogues(torch, dtype)
    finally:
        B.gemm_tile_override(prev)


def _gemm_epilogues(torch, dtype):
    M, N, K = 320, 448, 192
    a_p, a = _rand((M, K), dtype, 3)
    w_p, w = _rand((N, K), dtype, 4, std=0.1)
    bias_p, bias = _rand((N,), dtype, 5, std=0.5)
    res_p, res = _rand((M, N), dtype, 6)
    acc = a @ w.T
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    tol = 1e-2 if dtype == "bf16" else 1e-5
    A, W, Bi, R = _dev(a_p), _dev(w_p), _dev(bias_p), _dev(res_p)
    c = torch.empty((M, N), dtype=tdt, device="cuda")
    aux = torch.empty((M, N), dtype=tdt, device="cuda")
    B.gemm(A, W, c, M, N, K, epilogue=B.EPI_BIAS, bias=Bi)
    torch.cuda.synchronize()
    assert rel_err(B.to_host_f64(c), acc + bias) < tol
    B.gemm(A, W, c, M, N, K, epilogue=B.EPI_BIAS_GELU, bias=Bi, aux=aux)
    torch.cuda.synchronize()
    assert rel_err(B.to_host_f64(aux), acc + bias) < tol
    assert rel_err(B.to_host_f64(c), oracle.gelu(acc + bias)) < tol
    B.gemm(A, W, c, M, N, K, epilogue=B.EPI_BIAS_RESID, bias=Bi, resid=R, aux=aux)
    torch.cuda.synchronize()
    assert rel_err(B.to_host_f64(aux), acc) < tol
    assert rel_err(B.to_host_f64(c), res + acc + bias) < tol
    B.gemm(A, W, c, M, N, K, epilogue=B.EPI_BIAS_RESID, bias=Bi, resid=R, aux=None)
    torch.cuda.synchronize()
    assert rel_err(B.to_host_f64(c), res + acc + bias) < tol
    u_p, u = _rand((M, N), dtype, 7, std=2.0)
    U = _dev(u_p)
    B.gemm(A, W, c, M, N, K, epilogue=B.EPI_GELU_BWD, aux=U)
    torch.cuda.synchronize()
    assert rel_err(B.to_host_f64(c), acc * oracle.gelu_grad(u)) < tol


# widths: the smallest (one 8-wide chunk, one active lane), ragged chunk counts,
# the workloads' widths and the largest the kernels take (8192)
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("h", [8, 256, 520, 1600, 3072, 6144, 8192])
def test_layernorm_fwd_bwd(dtype, h):
    torch = need_gpu()
    print(f"[layernorm] {dtype} h={h}", flush=True)
    rows = 203  # a partial workgroup of rows and a partial 64-row reduction segment
    x_p, x = _rand((rows, h), dtype, 8, std=2.0, mean=0.5)
    g_p, g = _rand((h,), dtype, 9, std=0.1, mean=1.0)
    b_p, b = _rand((h,), dtype, 10, std=0.1)
    do_p, do = _rand((rows, h), dtype, 11)
    dr_p, dr = _rand((rows, h), dtype, 12)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    X = _dev(x_p)
    y = torch.empty((rows, h), dtype=tdt, device="cuda")
    mean = torch.empty(rows, dtype=torch.float32, device="cuda")
    rstd = torch.empty(rows, dtype=torch.float32, device="cuda")
    B.layernorm_fwd(X, _dev(g_p), _dev(b_p), y, mean, rstd, eps=1e-5)
    ref, xhat, rs = oracle.layer_norm_forward(x, g, b, 1e-5)
    dx = torch.empty((rows, h), dtype=tdt, device="cuda")
    dg = torch.empty(h, dtype=torch.float32, device="cuda")
    db = torch.empty(h, dtype=torch.float32, device="cuda")
    scratch = torch.empty(2 * B.reduce_scratch_elems(rows, h), dtype=torch.float32, device="cuda")
    B.layernorm_bwd(_dev(do_p), X, mean, rstd, _dev(g_p), _dev(dr_p), dx, dg, db, scratch)
    torch.cuda.synchronize()
    dz, dgr, dbr = oracle.layer_norm_backward(do, xhat, rs, g)
    tol = 1e-2 if dtype == "bf16" else 1e-5
    assert rel_err(B.to_host_f64(y), ref) < tol
    assert rel_err(rstd.cpu().numpy(), rs[:, 0]) < 1e-5
    assert rel_err(B.to_host_f64(dx), dr + dz) < tol
    assert rel_err(dg.cpu().numpy(), dgr) < 1e-4
    assert rel_err(db.cpu().numpy(), dbr) < 1e-5


# one row of one 8-column chunk, a ragged column count over a partial
# reduction segment, and a width past one workgroup's 512 columns
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("rows,cols", [(1, 8), (1000, 776), (8192, 3072)])
def test_column_sum(dtype, rows, cols):
    torch = need_gpu()
    print(f"[column sum] {dtype} {rows}x{cols}", flush=True)
    x_p, x = _rand((rows, cols), dtype, 13)
    out = torch.empty(cols, dtype=torch.float32, device="cuda")
    scratch = torch.empty(B.reduce_scratch_elems(rows, cols), dtype=torch.float32, device="cuda")
    B.column_sum(_dev(x_p), out, scratch)
    B.column_sum(_dev(x_p), out, scratch, accumulate=True)
    torch.cuda.synchronize()
    assert rel_err(out.cpu().numpy(), 2 * x.sum(0)) < 1e-5


ATTN_CASES = [(dt, d, s, 2, 3) for dt in ("bf16", "fp32") for d in (64, 96, 128) for s in (128, 320)]
ATTN_CASES += [("bf16", 128, 2048, 1, 2), ("bf16", 96, 1024, 2, 2)]  # full-length rows of the workloads
ATTN_CASES += [("bf16", d, 64, 2, 3) for d in (64, 96, 128)]  # one block: the pair's second half is empty


@pytest.mark.parametrize("dtype,d,seq,batch,heads", ATTN_CASES)
def test_attention_fwd_bwd(dtype, d, seq, batch, heads):
    torch = need_gpu()
    print(f"[attention] {dtype} d={d} seq={seq}", flush=True)
    qkv_p, qkv = _rand((batch, seq, 3, heads, d), dtype, 14 + d + seq)
    do_p, do = _rand((batch, seq, heads, d), dtype, 15 + d + seq)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    QKV = _dev(qkv_p)
    o = torch.empty((batch, seq, heads, d), dtype=tdt, device="cuda")
    lse = torch.empty((batch, heads, seq), dtype=torch.float32, device="cuda")
    B.attention_fwd(QKV, o, lse, batch, seq, heads, d)
    dqkv = torch.empty_like(QKV)
    delta = torch.empty((batch, heads, seq), dtype=torch.float32, device="cuda")
    B.attention_bwd(QKV, o, lse, _dev(do_p), dqkv, delta, batch, seq, heads, d)
    torch.cuda.synchronize()
    q, k, v = qkv[:, :, 0], qkv[:, :, 1], qkv[:, :, 2]
    O, P = oracle.causal_attention_forward(q, k, v)
    S = np.einsum("bihd,bjhd->bhij", q, k) / np.sqrt(d)
    S = np.where(np.triu(np.ones((seq, seq), bool), 1), -np.inf, S)
    m = S.max(-1, keepdims=True)
    lse_ref = (m + np.log(np.exp(S - m).sum(-1, keepdims=True)))[..., 0]
    tol = 2e-2 if dtype == "bf16" else 1e-5
    assert rel_err(B.to_host_f64(o), O) < tol
    assert np.max(np.abs(lse.cpu().numpy() - lse_ref)) < (2e-2 if dtype == "bf16" else 1e-5)
    # backward against the oracle with the GPU's own (rounded) forward output
    dq, dk, dv = oracle.causal_attention_backward(do, q, k, v, P)
    g = B.to_host_f64(dqkv)
    assert rel_err(g[:, :, 0], dq) < tol
    assert rel_err(g[:, :, 1], dk) < tol
    assert rel_err(g[:, :, 2], dv) < tol


@pytest.mark.parametrize("cfg", list(range(1, 11)))
@pytest.mark.parametrize("a_t,b_t", [(0, 0), (0, 1), (1, 1), (1, 0)])
@pytest.mark.parametrize("K", [64, 192, 320])
def test_gemm_every_tile_shape(cfg, a_t, b_t, K):
    """Each tile shape of the bf16 kernel on a ragged problem (M, N not
    multiples of 128 or 256), fp32 output so the check is tight.  K spans 1,
    3 or 5 stages of 64: fewer stages than the LDS ring holds, as many as a
    3-stage ring, and more, so that every path of the load schedule (loads
    issued in the prologue only, split over the two sub-steps after a
    barrier, none for the last stages) runs."""
    torch = need_gpu()
    M, N = 320, 448
    print(f"[gemm tile {cfg}] a_t={a_t} b_t={b_t} K={K}", flush=True)
    a_p, a = _rand((K, M) if a_t else (M, K), "bf16", 21)
    b_p, b = _rand((K, N) if b_t else (N, K), "bf16", 22)
    ref = (a.T if a_t else a) @ (b if b_t else b.T)
    c32 = torch.empty((M, N), dtype=torch.float32, device="cuda")
    prev = B.gemm_tile_override(cfg)
    try:
        B.gemm(_dev(a_p), _dev(b_p), c32, M, N, K, a_trans=a_t, b_trans=b_t, epilogue=B.EPI_F32, dtype=B.BF16)
        torch.cuda.synchronize()
    finally:
        B.gemm_tile_override(prev)
    assert rel_err(c32.cpu().numpy(), ref) < 2e-5


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("n", [0, 5, 4099, (1 << 20) + 7])
def test_count_nonfinite(dtype, n):
    """NaN and +-Inf planted at seeded positions (the ragged tail included),
    beside the largest finite values and subnormals, are counted exactly."""
    torch = need_gpu()
    print(f"[nonfinite] {dtype} n={n}", flush=True)
    rng = np.random.default_rng(90 + n)
    v = rng.standard_normal(n).astype(np.float32)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    big = float(torch.finfo(tdt).max)
    tiny = float(torch.finfo(tdt).tiny) / 4  # subnormal
    if n:
        idx = rng.choice(n, size=min(n, 37), replace=False)
        kinds = [np.nan, np.inf, -np.inf, big, -big, tiny]
        for j, i in enumerate(idx):
            v[i] = kinds[j % len(kinds)]
        v[n - 1] = np.nan  # the last element sits in the tail for most n
    x = torch.from_numpy(v).to(tdt).to("cuda")
    expect = int((~torch.isfinite(x.cpu().float())).sum().item())
    count = torch.full((1,), -1, dtype=torch.int64, device="cuda")
    B.count_nonfinite(x, count)
    torch.cuda.synchronize()
    assert int(count.item()) == expect
    # a second call overwrites the count rather than adding to it
    B.count_nonfinite(x, count)
    torch.cuda.synchronize()
    assert int(count.item()) == expect
