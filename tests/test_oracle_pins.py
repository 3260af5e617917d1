"""Pins of the fp64 oracle against what mathematics and library routines fix.

Each test states which part of the oracle it pins and how a plausible mistake
there (dropped term, wrong sign/index, transposed operand) would fail it.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2206_04959_amd import synth
from tests.oracle_helpers import f64_params, full_stage, local_stage, rel_max_err

EPS = 1e-5

# A shape small enough for finite differences over every parameter.
FD_SHAPE = synth.StageShape("fd", n_blocks=2, hidden=32, n_heads=2, ffn=128, seq_len=8,
                            micro_batch=2, tp_degree=1, dtype="fp32", x_std=1.0, w_std=0.2,
                            seed=7)


def _loss_and_grads(x, dy, blocks, nh_local):
    y, caches = oracle.stage_forward(x, blocks, nh_local, EPS)
    dx, grads, _ = oracle.stage_backward(dy, caches, blocks)
    return float((y * dy).sum()), dx, grads


def _loss(x, dy, blocks, nh_local):
    y, _ = oracle.stage_forward(x, blocks, nh_local, EPS)
    return float((y * dy).sum())


@pytest.mark.parametrize("t", [1, 2])
def test_p1_finite_differences_every_gradient(t):
    """P1: the directional derivative of <y, dy> along a random direction matches
    the oracle's gradient for the stage input and every parameter of every rank
    (a dropped term, sign or transposition anywhere in the backward fails)."""
    shape = FD_SHAPE.replace(tp_degree=t)
    full = full_stage(shape)
    blocks = [[oracle.shard_block(fb, r, t, shape.n_heads) for r in range(t)] for fb in full]
    nh = shape.local_heads
    x = synth.stage_input(shape).f64
    dy = synth.upstream_grad(shape).f64
    _, dx, grads = _loss_and_grads(x, dy, blocks, nh)
    rng = np.random.default_rng(11)
    h = 1e-5

    def check(analytic, perturb):
        v = rng.standard_normal(analytic.shape)
        lp = perturb(+h * v)
        lm = perturb(-h * v)
        fd = (lp - lm) / (2 * h)
        an = float((analytic * v).sum())
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (fd, an)

    check(dx, lambda dv: _loss(x + dv, dy, blocks, nh))
    for l in range(shape.n_blocks):
        for r in range(t):
            for name in synth.PARAM_NAMES:
                if name in ("ln1_g", "ln1_b", "b_o", "ln2_g", "ln2_b", "b2") and r > 0:
                    continue  # replicated: read from rank 0 in the reduced model

                def perturb(dv, l=l, r=r, name=name):
                    pb = [[dict(p) for p in shards] for shards in blocks]
                    pb[l][r][name] = pb[l][r][name] + dv
                    return _loss(x, dy, pb, nh)
                check(grads[l][r][name], perturb)


def test_p1_gelu_and_layernorm_derivatives_by_finite_differences():
    u = np.linspace(-6, 6, 241)
    h = 1e-6
    fd = (oracle.gelu(u + h) - oracle.gelu(u - h)) / (2 * h)
    assert np.max(np.abs(fd - oracle.gelu_grad(u))) < 1e-8
    rng = np.random.default_rng(3)
    z = rng.standard_normal((3, 5, 16)) * 2 + 0.5
    g = rng.standard_normal(16)
    bta = rng.standard_normal(16)
    dout = rng.standard_normal((3, 5, 16))
    _, xhat, rstd = oracle.layer_norm_forward(z, g, bta, EPS)
    dz, dg, db = oracle.layer_norm_backward(dout, xhat, rstd, g)
    v = rng.standard_normal(z.shape)
    f = lambda zz: float((oracle.layer_norm_forward(zz, g, bta, EPS)[0] * dout).sum())
    fd = (f(z + h * v) - f(z - h * v)) / (2 * h)
    assert abs(fd - float((dz * v).sum())) < 1e-7 * max(1, abs(fd))


def test_p2_softmax_invariants():
    """P2: rows of P sum to 1, P is exactly zero above the diagonal, P[0,0] = 1 so
    O[row 0] = v[row 0] exactly (a wrong mask direction or normalisation axis fails)."""
    rng = np.random.default_rng(5)
    b, s, nh, d = 2, 17, 3, 8
    q, k, v = (rng.standard_normal((b, s, nh, d)) * 3 for _ in range(3))
    O, P = oracle.causal_attention_forward(q, k, v)
    assert np.max(np.abs(P.sum(-1) - 1)) < 1e-12
    iu = np.triu_indices(s, 1)
    assert np.all(P[:, :, iu[0], iu[1]] == 0.0)
    assert np.all(P[:, :, 0, 0] == 1.0)
    assert np.array_equal(O[:, 0], v[:, 0])
    assert np.all(P >= 0)


def test_p3_zero_query_gives_prefix_mean():
    """P3: with q = 0 every unmasked logit is 0, so O_i is the mean of v_0..v_i."""
    rng = np.random.default_rng(6)
    b, s, nh, d = 2, 9, 2, 4
    k = rng.standard_normal((b, s, nh, d))
    v = rng.standard_normal((b, s, nh, d))
    O, _ = oracle.causal_attention_forward(np.zeros_like(k), k, v)
    prefix = np.cumsum(v, axis=1) / np.arange(1, s + 1)[None, :, None, None]
    assert np.max(np.abs(O - prefix)) < 1e-13


def test_p3_layernorm_pre_affine_moments_and_gelu_identities():
    rng = np.random.default_rng(8)
    z = rng.standard_normal((4, 7, 33)) * 5 + 3
    _, xhat, rstd = oracle.layer_norm_forward(z, np.ones(33), np.zeros(33), 0.0)
    assert np.max(np.abs(xhat.mean(-1))) < 1e-13
    assert np.max(np.abs((xhat ** 2).mean(-1) - 1)) < 1e-12   # biased variance
    u = np.linspace(-5, 5, 101)
    assert oracle.gelu(np.array(0.0)) == 0.0
    # 0.5 u (1 + tanh(w)) - 0.5 (-u)(1 + tanh(-w)) = u for the odd inner w(u)
    assert np.max(np.abs(oracle.gelu(u) - oracle.gelu(-u) - u)) < 1e-14
    # large |u|: gelu -> relu
    assert abs(oracle.gelu(np.array(30.0)) - 30.0) < 1e-12
    assert abs(oracle.gelu(np.array(-30.0))) < 1e-12


def test_p3_bias_gradients_are_token_sums():
    shape = FD_SHAPE
    blocks = [[p] for p in local_stage(shape)]
    x = synth.stage_input(shape).f64
    dy = synth.upstream_grad(shape).f64
    y, caches = oracle.stage_forward(x, blocks, shape.local_heads, EPS)
    _, grads, bwd = oracle.stage_backward(dy, caches, blocks)
    last = shape.n_blocks - 1
    assert np.allclose(grads[last][0]["b2"], dy.sum(axis=(0, 1)), rtol=0, atol=1e-12)
    assert np.allclose(grads[last][0]["b_o"], bwd[last]["dx1"].sum(axis=(0, 1)), rtol=0, atol=1e-12)


def _torch_block(x, p, n_heads, eps):
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    h = x.shape[-1]
    ln1 = F.layer_norm(x, (h,), p["ln1_g"], p["ln1_b"], eps)
    qkv = F.linear(ln1, p["w_qkv"], p["b_qkv"])
    b, s, _ = x.shape
    d = h // n_heads
    q, k, v = (qkv[..., i * h:(i + 1) * h].reshape(b, s, n_heads, d).transpose(1, 2) for i in range(3))
    o = F.scaled_dot_product_attention(q, k, v, is_causal=True)
    o = o.transpose(1, 2).reshape(b, s, h)
    x1 = x + F.linear(o, p["w_o"], p["b_o"])
    ln2 = F.layer_norm(x1, (h,), p["ln2_g"], p["ln2_b"], eps)
    g = F.gelu(F.linear(ln2, p["w1"], p["b1"]), approximate="tanh")
    return x1 + F.linear(g, p["w2"], p["b2"])


def test_p6_torch_fp64_autograd_whole_stage():
    """P6: library special case: the t = 1 stage equals torch's fp64 LayerNorm /
    Linear / causal scaled-dot-product attention / tanh-GeLU composition, forward
    and every gradient."""
    torch = pytest.importorskip("torch")
    shape = synth.StageShape("p6", n_blocks=2, hidden=64, n_heads=4, ffn=256, seq_len=16,
                             micro_batch=2, dtype="fp32", x_std=1.0, w_std=0.1, seed=9)
    params = local_stage(shape)
    x = synth.stage_input(shape).f64
    dy = synth.upstream_grad(shape).f64
    res = oracle.shard_run(x, dy, params, shape.local_heads, EPS)

    tx = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    tp = [{k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in p.items()} for p in params]
    h = tx
    for p in tp:
        h = _torch_block(h, p, shape.n_heads, EPS)
    h.backward(torch.tensor(dy))
    assert rel_max_err(res["y"], h.detach().numpy()) < 1e-12
    assert rel_max_err(res["dx"], tx.grad.numpy()) < 1e-10
    for l, p in enumerate(tp):
        for name in synth.PARAM_NAMES:
            assert rel_max_err(res["grads"][l][name], p[name].grad.numpy()) < 1e-10, (l, name)


@pytest.mark.parametrize("t", [2, 4])
def test_p4_tensor_parallel_reassembly(t):
    """P4: summing the t ranks' partial sums reproduces the full (t = 1) block:
    forward partials, backward partials, outputs and gradient slices (a wrong head
    or FFN-unit map, or a bias added per rank, fails)."""
    shape = synth.StageShape("p4", n_blocks=1, hidden=64, n_heads=8, ffn=256, seq_len=12,
                             micro_batch=2, dtype="fp32", x_std=1.0, w_std=0.1, seed=10)
    full = full_stage(shape)[0]
    x = synth.stage_input(shape).f64
    dy = synth.upstream_grad(shape).f64
    y1, c1 = oracle.block_forward(x, [full], shape.n_heads, EPS)
    dx1, g1, b1 = oracle.block_backward(dy, c1, [full])
    shards = [oracle.shard_block(full, r, t, shape.n_heads) for r in range(t)]
    yt, ct = oracle.block_forward(x, shards, shape.n_heads // t, EPS)
    dxt, gt, bt = oracle.block_backward(dy, ct, shards)
    assert rel_max_err(yt, y1) < 1e-12
    assert rel_max_err(dxt, dx1) < 1e-12
    assert rel_max_err(sum(ct["p_o"]), c1["p_o"][0]) < 1e-12
    assert rel_max_err(sum(ct["p_f"]), c1["p_f"][0]) < 1e-12
    assert rel_max_err(sum(bt["d_ln1"]), b1["d_ln1"][0]) < 1e-12
    assert rel_max_err(sum(bt["d_ln2"]), b1["d_ln2"][0]) < 1e-12
    for r in range(t):
        sliced = oracle.shard_block(g1[0], r, t, shape.n_heads)
        for name in synth.PARAM_NAMES:
            assert rel_max_err(gt[r][name], sliced[name]) < 1e-11, (r, name)


@pytest.mark.parametrize("t,rank", [(2, 1), (4, 2)])
def test_p5_identity_reduce_equals_zero_padded_full_model(t, rank):
    """P5: one shard with R = identity (what one GPU computes) over a whole stage
    equals the full model whose other ranks' column-parallel weights are zero."""
    shape = synth.StageShape("p5", n_blocks=3, hidden=64, n_heads=8, ffn=256, seq_len=10,
                             micro_batch=2, tp_degree=t, dtype="fp32", x_std=1.0, w_std=0.1,
                             seed=12)
    local = local_stage(shape, rank)
    x = synth.stage_input(shape).f64
    dy = synth.upstream_grad(shape).f64
    res = oracle.shard_run(x, dy, local, shape.local_heads, EPS)
    padded = [oracle.zero_pad_block(p, rank, t) for p in local]
    full = oracle.shard_run(x, dy, padded, shape.n_heads, EPS)
    assert rel_max_err(res["y"], full["y"]) < 1e-12
    assert rel_max_err(res["dx"], full["dx"]) < 1e-12
    for l in range(shape.n_blocks):
        assert rel_max_err(res["p_o"][l], full["p_o"][l]) < 1e-12
        assert rel_max_err(res["p_f"][l], full["p_f"][l]) < 1e-12
        assert rel_max_err(res["d_ln1"][l], full["d_ln1"][l]) < 1e-12
        assert rel_max_err(res["d_ln2"][l], full["d_ln2"][l]) < 1e-12
        sliced = oracle.shard_block(full["grads"][l], rank, t, shape.n_heads)
        for name in synth.PARAM_NAMES:
            assert rel_max_err(res["grads"][l][name], sliced[name]) < 1e-11, (l, name)


def test_p7_sub_micro_batch_split_is_independent():
    """P7: the sub-micro-batches are independent: per-slice forwards concatenate to
    the unsplit forward and per-slice weight gradients sum to the unsplit ones."""
    shape = synth.StageShape("p7", n_blocks=2, hidden=64, n_heads=4, ffn=256, seq_len=12,
                             micro_batch=4, dtype="fp32", x_std=1.0, w_std=0.1, seed=13)
    params = local_stage(shape)
    x = synth.stage_input(shape).f64
    dy = synth.upstream_grad(shape).f64
    whole = oracle.shard_run(x, dy, params, shape.local_heads, EPS)
    n = 2
    m = shape.micro_batch // n
    parts = [oracle.shard_run(x[j * m:(j + 1) * m], dy[j * m:(j + 1) * m], params,
                              shape.local_heads, EPS) for j in range(n)]
    assert rel_max_err(np.concatenate([p["y"] for p in parts]), whole["y"]) < 1e-13
    assert rel_max_err(np.concatenate([p["dx"] for p in parts]), whole["dx"]) < 1e-13
    for l in range(shape.n_blocks):
        for name in synth.PARAM_NAMES:
            assert rel_max_err(sum(p["grads"][l][name] for p in parts), whole["grads"][l][name]) < 1e-12
