"""Pin P4 on the GPU: the tensor-parallel shard map reassembles the full block.

t ranks' shards of one full (t = 1) block are cut here by the layout the C
header documents (rank r owns heads [r a/t, (r+1) a/t): its QKV rows are its q
rows, then its k rows, then its v rows, and its W_o columns are those heads'
channels; it owns FFN units [r f/t, (r+1) f/t): W1 rows, b1, W2 columns;
LayerNorms, b_o and b2 are replicated).  Every rank's shard then runs through
the library on the one GPU, and the host sums the ranks' partial results where
tensor parallelism would run an AllReduce (paper Sec. 2, "Tensor model
parallelism"; two AllReduces per block in the forward pass and two in the
backward pass, Sec. 5.3).  The summed partials, the block output, the block's
input gradient and every rank's weight gradients must equal the full block of
the fp64 oracle (t = 1, nothing sharded) within the stated tolerances.

Two routes:
* rank by rank through the per-kernel entry points (GEMM, attention,
  LayerNorm), with the host sums between the steps, so that every partial of
  the block (p_o, p_f, d_ln2, d_ln1) is checked after its own reduction;
* the stage entry point itself, one handle per rank: the first partial of the
  first block (p_o) depends only on the stage input, so the ranks' hand-off
  buffers must sum to the full block's p_o.  (Later partials of a one-GPU
  stage see R = identity instead of the sum, so only this one reassembles.)
"""
import numpy as np
import pytest

import oracle
from paper_2206_04959_amd import binding as B
from paper_2206_04959_amd import synth
from tests.gpu_util import need_gpu, rel_err, tol_for

pytestmark = pytest.mark.gpu

# Small blocks spanning several GEMM and attention tiles, every head_dim.
CASES = {
    "d64-t2": synth.StageShape("p4a", n_blocks=1, hidden=512, n_heads=8, ffn=2048, seq_len=128, micro_batch=2,
                               tp_degree=2, seed=41),
    "d64-t4": synth.StageShape("p4b", n_blocks=1, hidden=512, n_heads=8, ffn=2048, seq_len=128, micro_batch=2,
                               tp_degree=4, seed=42),
    "d96-t2": synth.StageShape("p4c", n_blocks=1, hidden=384, n_heads=4, ffn=1536, seq_len=192, micro_batch=2,
                               tp_degree=2, seed=43),
    "d128-t4": synth.StageShape("p4d", n_blocks=1, hidden=1024, n_heads=8, ffn=4096, seq_len=128, micro_batch=2,
                                tp_degree=4, seed=44),
}


def cut(full, r, t):
    """Rank r's shard of a full block (any array type: fp64 values or device payload)."""
    h = full["w_o"].shape[0]
    f = full["w1"].shape[0]
    hl, fl = h // t, f // t
    rows = np.concatenate([np.arange(part * h + r * hl, part * h + (r + 1) * hl) for part in range(3)])
    out = {k: full[k] for k in ("ln1_g", "ln1_b", "b_o", "ln2_g", "ln2_b", "b2")}
    out["w_qkv"] = full["w_qkv"][rows]
    out["b_qkv"] = full["b_qkv"][rows]
    out["w_o"] = full["w_o"][:, r * hl:(r + 1) * hl]
    out["w1"] = full["w1"][r * fl:(r + 1) * fl]
    out["b1"] = full["b1"][r * fl:(r + 1) * fl]
    out["w2"] = full["w2"][:, r * fl:(r + 1) * fl]
    return {k: np.ascontiguousarray(v) for k, v in out.items()}


def device_round(v64, dtype):
    """What an AllReduce in the activation dtype hands back: the sum rounded to it."""
    if dtype == "bf16":
        bits = synth.f32_to_bf16_bits(v64.astype(np.float32))
        return bits
    return v64.astype(np.float32)


def full_reference(shape):
    full = synth.full_block_params(shape, 0)
    x, dy = synth.stage_input(shape), synth.upstream_grad(shape)
    ref = oracle.shard_run(x.f64, dy.f64, [{k: v.f64 for k, v in full.items()}], shape.n_heads, shape.ln_eps)
    return full, x, dy, ref


def rank_by_rank(shape, full, x_h, dy_h):
    """The block through the per-kernel entry points, rank by rank, host sums at
    each AllReduce.  Returns the reassembled values and every rank's weight
    gradients."""
    torch = need_gpu()
    t, h, a, d = shape.tp_degree, shape.hidden, shape.n_heads, shape.head_dim
    b, s, T = shape.micro_batch, shape.seq_len, shape.tokens
    hl, fl, al = h // t, shape.ffn // t, a // t
    dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    dev = lambda p: B.to_device(np.ascontiguousarray(p))  # noqa: E731
    host = lambda g: B.to_host_f64(g)  # noqa: E731
    empty = lambda *shp, dtype=dt: torch.empty(shp, dtype=dtype, device="cuda")  # noqa: E731
    ranks = [{k: dev(v) for k, v in cut({k: v.payload for k, v in full.items()}, r, t).items()} for r in range(t)]
    rep = ranks[0]
    x = dev(x_h.payload).reshape(T, h)
    dy = dev(dy_h.payload).reshape(T, h)
    out = {}

    # attention block, forward
    ln1, mu1, rs1 = empty(T, h), empty(T, dtype=torch.float32), empty(T, dtype=torch.float32)
    B.layernorm_fwd(x, rep["ln1_g"], rep["ln1_b"], ln1, mu1, rs1, eps=shape.ln_eps)
    per = []
    for p in ranks:
        qkv = empty(T, 3 * hl)
        B.gemm(ln1, p["w_qkv"], qkv, T, 3 * hl, h, epilogue=B.EPI_BIAS, bias=p["b_qkv"])
        o, lse = empty(T, hl), empty(b, al, s, dtype=torch.float32)
        B.attention_fwd(qkv, o, lse, b, s, al, d)
        po = empty(T, h)
        B.gemm(o, p["w_o"], po, T, h, hl)
        per.append(dict(qkv=qkv, o=o, lse=lse, po=po))
    torch.cuda.synchronize()
    out["p_o"] = sum(host(c["po"]) for c in per)
    x1_64 = x_h.f64.reshape(T, h) + out["p_o"] + full["b_o"].f64
    x1 = dev(device_round(x1_64, shape.dtype))

    # FFN block, forward
    ln2, mu2, rs2 = empty(T, h), empty(T, dtype=torch.float32), empty(T, dtype=torch.float32)
    B.layernorm_fwd(x1, rep["ln2_g"], rep["ln2_b"], ln2, mu2, rs2, eps=shape.ln_eps)
    for p, c in zip(ranks, per):
        u, g = empty(T, fl), empty(T, fl)
        B.gemm(ln2, p["w1"], g, T, fl, h, epilogue=B.EPI_BIAS_GELU, bias=p["b1"], aux=u)
        pf = empty(T, h)
        B.gemm(g, p["w2"], pf, T, h, fl)
        c.update(u=u, g=g, pf=pf)
    torch.cuda.synchronize()
    out["p_f"] = sum(host(c["pf"]) for c in per)
    out["y"] = host(x1) + out["p_f"] + full["b2"].f64

    # FFN block, backward
    for p, c in zip(ranks, per):
        du = empty(T, fl)
        B.gemm(dy, p["w2"], du, T, fl, h, b_trans=True, epilogue=B.EPI_GELU_BWD, aux=c["u"])
        dln2 = empty(T, h)
        B.gemm(du, p["w1"], dln2, T, h, fl, b_trans=True)
        c.update(du=du, dln2=dln2)
    torch.cuda.synchronize()
    out["d_ln2"] = sum(host(c["dln2"]) for c in per)
    d_ln2 = dev(device_round(out["d_ln2"], shape.dtype))
    scratch = empty(2 * B.reduce_scratch_elems(T, h), dtype=torch.float32)
    dg, db = empty(h, dtype=torch.float32), empty(h, dtype=torch.float32)
    dx1 = empty(T, h)
    B.layernorm_bwd(d_ln2, x1, mu2, rs2, rep["ln2_g"], dy, dx1, dg, db, scratch)

    # attention block, backward
    for p, c in zip(ranks, per):
        do = empty(T, hl)
        B.gemm(dx1, p["w_o"], do, T, hl, h, b_trans=True)
        dqkv, delta = empty(T, 3 * hl), empty(b, al, s, dtype=torch.float32)
        B.attention_bwd(c["qkv"], c["o"], c["lse"], do, dqkv, delta, b, s, al, d)
        dln1 = empty(T, h)
        B.gemm(dqkv, p["w_qkv"], dln1, T, h, 3 * hl, b_trans=True)
        c.update(dqkv=dqkv, dln1=dln1)
    torch.cuda.synchronize()
    out["d_ln1"] = sum(host(c["dln1"]) for c in per)
    d_ln1 = dev(device_round(out["d_ln1"], shape.dtype))
    dx = empty(T, h)
    B.layernorm_bwd(d_ln1, x, mu1, rs1, rep["ln1_g"], dx1, dx, dg, db, scratch)

    # every rank's weight gradients (dW = dY^T X over all tokens)
    grads = []
    for c in per:
        gr = {}
        for name, dyv, xv, n_out, n_in in (("w2", dy, c["g"], h, fl), ("w1", c["du"], ln2, fl, h),
                                            ("w_o", dx1, c["o"], h, hl), ("w_qkv", c["dqkv"], ln1, 3 * hl, h)):
            w = empty(n_out, n_in, dtype=torch.float32)
            B.gemm(dyv, xv, w, n_out, n_in, T, a_trans=True, b_trans=True, epilogue=B.EPI_F32, dtype=B._dt(dyv))
            gr[name] = w
        grads.append(gr)
    torch.cuda.synchronize()
    out["dx"] = host(dx)
    out["grads"] = [{k: v.cpu().numpy().astype(np.float64) for k, v in gr.items()} for gr in grads]
    return out


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("name", sorted(CASES))
def test_ranks_reassemble_the_full_block(name, dtype):
    shape = CASES[name].replace(dtype=dtype, x_std=1.0)
    print(f"[tp reassembly] {name} {dtype}: {shape}", flush=True)
    full, x, dy, ref = full_reference(shape)
    got = rank_by_rank(shape, full, x, dy)
    t = shape.tp_degree
    errs = {"y": rel_err(got["y"].reshape(ref["y"].shape), ref["y"]),
            "dx": rel_err(got["dx"].reshape(ref["dx"].shape), ref["dx"])}
    for k in ("p_o", "p_f", "d_ln1", "d_ln2"):
        errs[k] = rel_err(got[k].reshape(ref[k][0].shape), ref[k][0])
    for r in range(t):
        want = cut(ref["grads"][0], r, t)
        for k, v in got["grads"][r].items():
            errs[f"{k}@{r}"] = rel_err(v, want[k])
    tol = tol_for(shape)
    worst = max(errs, key=errs.get)
    print(f"  worst {worst} = {errs[worst]:.3e} (tolerance {tol})", flush=True)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad


@pytest.mark.parametrize("name", ["d64-t4", "d96-t2"])
def test_stage_hand_off_buffers_reassemble_first_partial(name):
    torch = need_gpu()
    shape = CASES[name].replace(dtype="bf16", x_std=1.0)
    full, x, dy, ref = full_reference(shape)
    t, T, h = shape.tp_degree, shape.tokens, shape.hidden
    xd = B.to_device(x.payload)
    total = np.zeros((shape.micro_batch, shape.seq_len, h))
    for r in range(t):
        cfg = B.make_config(shape)
        params = B.to_device(B.pack_params(cfg, [cut({k: v.payload for k, v in full.items()}, r, t)]))
        y = torch.empty_like(xd)
        fp = torch.empty((1, 2, T * h), dtype=xd.dtype, device="cuda")
        st = B.Stage(shape)
        st.fwd(params, xd, y, fp)
        torch.cuda.synchronize()
        total += B.to_host_f64(fp[0, 0]).reshape(total.shape)
        st.close()
    e = rel_err(total, ref["p_o"][0])
    print(f"[stage hand-off reassembly] {name}: p_o error {e:.3e}", flush=True)
    assert e <= tol_for(shape)
