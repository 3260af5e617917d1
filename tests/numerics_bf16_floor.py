"""Study (not a test): the bf16 floor of the max-relative error metric.

Re-runs the oracle's stage with bf16 round-to-nearest applied at the points
where the HIP path stores a bf16 tensor (every GEMM/attention operand, the
residual stream, the gradient chain), and reports the max-relative error of y,
dx and the LN1 input-gradient partials against the exact oracle, for all
rounding points and for subsets.  It shows how much error bf16 storage alone
produces for a workload, independent of any kernel.

    python tests/numerics_bf16_floor.py [preset] [micro_batch]
"""
import math
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import numpy as np  # noqa: E402

import oracle  # noqa: E402
from paper_2206_04959_amd import synth  # noqa: E402


def rb(a):  # round to bf16
    a32 = np.asarray(a, dtype=np.float32)
    return synth.bf16_bits_to_f64(synth.f32_to_bf16_bits(a32)).reshape(a32.shape)


def fwd_block(x, p, nh, eps, R):
    r = lambda name, v: rb(v) if name in R else v
    ln1, xh1, rs1 = oracle.layer_norm_forward(x, p["ln1_g"], p["ln1_b"], eps); ln1r = r("ln1", ln1)
    qkv = r("qkv", ln1r @ p["w_qkv"].T + p["b_qkv"])
    b, s, _ = x.shape; hl = qkv.shape[-1] // 3; d = hl // nh
    q = qkv[..., :hl].reshape(b, s, nh, d); k = qkv[..., hl:2*hl].reshape(b, s, nh, d); v = qkv[..., 2*hl:].reshape(b, s, nh, d)
    O4, P = oracle.causal_attention_forward(q, k, v)
    if "P_fwd" in R: O4 = (rb(P) @ v.transpose(0, 2, 1, 3)).transpose(0, 2, 1, 3)
    O = r("O", O4.reshape(b, s, hl))
    po = O @ p["w_o"].T
    x1 = r("x1", x + po + p["b_o"])
    ln2, xh2, rs2 = oracle.layer_norm_forward(x1, p["ln2_g"], p["ln2_b"], eps); ln2r = r("ln2", ln2)
    u = ln2r @ p["w1"].T + p["b1"]; ur = r("u", u); g = r("g", oracle.gelu(u))
    y = r("y", x1 + g @ p["w2"].T + p["b2"])
    return y, dict(x=x, xh1=xh1, rs1=rs1, ln1=ln1r, q=q, k=k, v=v, P=P, O=O, x1=x1, xh2=xh2, rs2=rs2, ln2=ln2r, u=ur, g=g, nh=nh, d=d)

def bwd_block(dy, c, p, R):
    r = lambda name, v: rb(v) if name in R else v
    b, s, h = dy.shape; nh, d = c["nh"], c["d"]; hl = nh * d
    du = r("du", (dy @ p["w2"]) * oracle.gelu_grad(c["u"]))
    dln2 = r("dln2", du @ p["w1"])
    dz2, _, _ = oracle.layer_norm_backward(dln2, c["xh2"], c["rs2"], p["ln2_g"])
    dx1 = r("dx1", dy + dz2)
    dO = r("dO", dx1 @ p["w_o"]).reshape(b, s, nh, d)
    qh, kh, vh, dOh = (t.transpose(0, 2, 1, 3) for t in (c["q"], c["k"], c["v"], dO))
    P = c["P"]; Pb = rb(P) if "P_bwd" in R else P
    dV = Pb.transpose(0, 1, 3, 2) @ dOh
    dP = dOh @ vh.transpose(0, 1, 3, 2)
    if "delta_bf16O" in R: delta = (dO * c["O"].reshape(b, s, nh, d)).sum(-1).transpose(0, 2, 1)[..., None]
    else: delta = (dP * P).sum(-1, keepdims=True)
    dS = P * (dP - delta)
    if "dS" in R: dS = rb(dS)
    dQ = (dS @ kh) / math.sqrt(d); dK = (dS.transpose(0, 1, 3, 2) @ qh) / math.sqrt(d)
    dqkv = r("dqkv", np.concatenate([t.transpose(0, 2, 1, 3).reshape(b, s, hl) for t in (dQ, dK, dV)], -1))
    dln1 = r("dln1", dqkv @ p["w_qkv"])
    dz1, _, _ = oracle.layer_norm_backward(dln1, c["xh1"], c["rs1"], p["ln1_g"])
    dx = r("dxchain", dx1 + dz1)
    return dx, dict(dln1=dln1, dln2=dln2)

def stage(x, dy, ps, nh, R):
    caches = []; h = x
    for p in ps:
        h, c = fwd_block(h, p, nh, 1e-5, R); caches.append(c)
    g = dy; outs = []
    for l in range(len(ps) - 1, -1, -1):
        g, o = bwd_block(g, caches[l], ps[l], R); outs.append(o)
    return h, g, outs[::-1]



ALL = {"ln1", "qkv", "P_fwd", "O", "x1", "ln2", "u", "g", "y", "du", "dln2", "dx1", "dO", "P_bwd", "delta_bf16O",
       "dS", "dqkv", "dln1", "dxchain"}
FWD = {"ln1", "qkv", "P_fwd", "O", "x1", "ln2", "u", "g", "y"}


def main():
    name = sys.argv[1] if len(sys.argv) > 1 else "gpt-20b-tp8"
    b = int(sys.argv[2]) if len(sys.argv) > 2 else 1
    shape = synth.PRESETS[name].replace(micro_batch=b, n_sub=1)
    ps = [{k: v.f64 for k, v in p.items()} for p in synth.stage_params(shape)]
    x = synth.stage_input(shape).f64
    dy = synth.upstream_grad(shape).f64
    y0, dx0, o0 = stage(x, dy, ps, shape.local_heads, set())

    def err(a, c):
        return np.max(np.abs(a - c)) / np.max(np.abs(c))

    variants = {"all bf16 points": ALL, "forward points only": FWD, "backward points only": ALL - FWD,
                "fp32 residual stream": ALL - {"x1", "y"}}
    for vname, R in variants.items():
        y1, dx1, o1 = stage(x, dy, ps, shape.local_heads, R)
        print(f"{vname:22s} y {err(y1, y0):.3e} dx {err(dx1, dx0):.3e} "
              + " ".join(f"dln1[{l}] {err(o1[l]['dln1'], o0[l]['dln1']):.3e}" for l in range(len(ps))), flush=True)


if __name__ == "__main__":
    main()
