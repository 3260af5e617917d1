"""Plain fp64 CPU oracle of one GPU's share of a GPT pipeline stage.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module; only the test suite, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code with the HIP library.

What it computes (the plain definition; every scheduling trick of the method
reaches exactly this result):

* A stage is a run of consecutive transformer blocks (Sec. 2 "Pipeline model
  parallelism"; Sec. 4.2: pipeline stages are continuous parts of the subgraph
  sequence); block l's output is block l+1's input.
* A block is a GPT decoder block made of an attention block and an FFN block
  (Sec. 5.3, first paragraph), split Megatron-style across t tensor-parallel
  ranks: weight matrices cut along rows or columns, with an AllReduce making the
  result correct (Sec. 2 "Tensor model parallelism"; Sec. 4.1: TMP follows
  Megatron-LM).  The FP carries two AllReduces per block and the BP two more
  (Sec. 5.3).  Here R denotes that reduction: the sum over ranks.
* Sub-micro-batches are even, mutually independent splits of the micro-batch
  (Sec. 5.3, sub-pipelined TMP), so splitting changes nothing in the result.
* Recomputation re-evaluates the same forward pass (Sec. 2 "Activation
  recomputation"; Sec. 5.2), so it changes nothing in the result either.

The paper leaves the block's internals unstated (LayerNorm placement, GeLU
form, biases, softmax scale and mask).  The readings used here: pre-LN GPT-2
block with biases on every linear layer, LayerNorm with biased variance and
eps inside the square root, GeLU in its tanh form, softmax scale 1/sqrt(d),
masked logits at -inf (the diagonal is never masked), no dropout; a
row-parallel layer's bias is added once, after R.

Layouts: activations are [b, s, features]; a weight is stored [out, in], so a
linear layer computes x @ W.T + b.  A rank's fused QKV output is laid out
[q | k | v], each part [local heads, head_dim].

Parity is pinned by the tests in ``tests/test_oracle_*.py`` (finite
differences, softmax invariants, closed-form special cases, torch fp64
autograd, brute-force tensor-parallel reassembly, zero-padding equivalence,
split independence).
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence

import numpy as np

GELU_C = math.sqrt(2.0 / math.pi)
GELU_A = 0.044715


# --------------------------------------------------------------------------
# Elementwise and row-wise pieces
# --------------------------------------------------------------------------

def layer_norm_forward(z, gamma, beta, eps):
    """LayerNorm over the last axis: gamma * (z - mean) / sqrt(var + eps) + beta,
    with the biased (divide-by-h) variance.  Returns (out, xhat, rstd)."""
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (z - mu) * rstd
    return gamma * xhat + beta, xhat, rstd


def layer_norm_backward(dout, xhat, rstd, gamma):
    """Reverse mode of ``layer_norm_forward``.  Returns (dz, dgamma, dbeta);
    the parameter gradients are summed over every token."""
    tok_axes = tuple(range(dout.ndim - 1))
    dgamma = (dout * xhat).sum(axis=tok_axes)
    dbeta = dout.sum(axis=tok_axes)
    dxhat = dout * gamma
    dz = rstd * (dxhat
                 - dxhat.mean(axis=-1, keepdims=True)
                 - xhat * (dxhat * xhat).mean(axis=-1, keepdims=True))
    return dz, dgamma, dbeta


def gelu(u):
    """GeLU, tanh form: 0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3)))."""
    return 0.5 * u * (1.0 + np.tanh(GELU_C * (u + GELU_A * u ** 3)))


def gelu_grad(u):
    """d gelu / d u for the tanh form above."""
    th = np.tanh(GELU_C * (u + GELU_A * u ** 3))
    return 0.5 * (1.0 + th) + 0.5 * u * (1.0 - th * th) * GELU_C * (1.0 + 3.0 * GELU_A * u * u)


# --------------------------------------------------------------------------
# Causal self-attention on a rank's local heads
# --------------------------------------------------------------------------

def causal_attention_forward(q, k, v):
    """q, k, v: [b, s, heads, d].  S = q k^T / sqrt(d) with S[i, j] = -inf for
    j > i, P = row softmax of S, O = P v.  Returns (O [b, s, heads, d], P [b, heads, s, s])."""
    d = q.shape[-1]
    s = q.shape[1]
    qh, kh, vh = (t.transpose(0, 2, 1, 3) for t in (q, k, v))  # [b, heads, s, d]
    S = (qh @ kh.transpose(0, 1, 3, 2)) / math.sqrt(d)
    future = np.triu(np.ones((s, s), dtype=bool), k=1)
    S = np.where(future, -np.inf, S)
    S = S - S.max(axis=-1, keepdims=True)
    E = np.exp(S)
    P = E / E.sum(axis=-1, keepdims=True)
    O = (P @ vh).transpose(0, 2, 1, 3)
    return O, P


def causal_attention_backward(dO, q, k, v, P):
    """Reverse mode of ``causal_attention_forward`` (softmax Jacobian written out)."""
    d = q.shape[-1]
    qh, kh, vh, dOh = (t.transpose(0, 2, 1, 3) for t in (q, k, v, dO))  # [b, heads, s, d]
    Pt = P.transpose(0, 1, 3, 2)
    dV = Pt @ dOh
    dP = dOh @ vh.transpose(0, 1, 3, 2)
    dS = P * (dP - (dP * P).sum(axis=-1, keepdims=True))
    dQ = (dS @ kh) / math.sqrt(d)
    dK = (dS.transpose(0, 1, 3, 2) @ qh) / math.sqrt(d)
    return tuple(t.transpose(0, 2, 1, 3) for t in (dQ, dK, dV))


# --------------------------------------------------------------------------
# One block, t ranks (a list of shards); R = sum over the list
# --------------------------------------------------------------------------

def _tok_outer(a, b):
    """sum over all tokens of a[t, i] * b[t, j] (a weight gradient dY^T X)."""
    return a.reshape(-1, a.shape[-1]).T @ b.reshape(-1, b.shape[-1])


def _split_heads(qkv, n_heads_local):
    b, s, three_hl = qkv.shape
    hl = three_hl // 3
    d = hl // n_heads_local
    q = qkv[..., 0 * hl:1 * hl].reshape(b, s, n_heads_local, d)
    k = qkv[..., 1 * hl:2 * hl].reshape(b, s, n_heads_local, d)
    v = qkv[..., 2 * hl:3 * hl].reshape(b, s, n_heads_local, d)
    return q, k, v


def block_forward(x, shards: Sequence[Dict[str, np.ndarray]], n_heads_local: int, eps: float):
    """Forward of one block given every rank's shard (one shard = the one-GPU case,
    where R is the identity).  Replicated parameters (LayerNorms, b_o, b2) are read
    from shard 0.  Returns (y, cache); cache['p_o'][r] and cache['p_f'][r] are rank
    r's row-parallel partial sums, the values each rank hands to the AllReduce."""
    p0 = shards[0]
    ln1, xhat1, rstd1 = layer_norm_forward(x, p0["ln1_g"], p0["ln1_b"], eps)
    per_rank = []
    p_o = []
    for p in shards:
        qkv = ln1 @ p["w_qkv"].T + p["b_qkv"]
        q, k, v = _split_heads(qkv, n_heads_local)
        O4, P = causal_attention_forward(q, k, v)
        O = O4.reshape(x.shape[0], x.shape[1], -1)
        p_o.append(O @ p["w_o"].T)
        per_rank.append({"qkv": qkv, "q": q, "k": k, "v": v, "P": P, "O": O})
    x1 = x + sum(p_o) + p0["b_o"]

    ln2, xhat2, rstd2 = layer_norm_forward(x1, p0["ln2_g"], p0["ln2_b"], eps)
    p_f = []
    for p, c in zip(shards, per_rank):
        u = ln2 @ p["w1"].T + p["b1"]
        g = gelu(u)
        p_f.append(g @ p["w2"].T)
        c.update(u=u, g=g)
    y = x1 + sum(p_f) + p0["b2"]

    cache = dict(x=x, ln1=ln1, xhat1=xhat1, rstd1=rstd1, x1=x1, ln2=ln2, xhat2=xhat2,
                 rstd2=rstd2, ranks=per_rank, p_o=p_o, p_f=p_f, n_heads_local=n_heads_local)
    return y, cache


def block_backward(dy, cache, shards: Sequence[Dict[str, np.ndarray]]):
    """Reverse mode of ``block_forward``.  Returns (dx, grads, bwd) where grads[r] is
    rank r's gradient dict (replicated parameters' gradients are identical on every
    rank), and bwd['d_ln2'][r], bwd['d_ln1'][r] are rank r's column-parallel input
    gradients (the partial sums handed to the backward AllReduces)."""
    p0 = shards[0]
    tok = (0, 1)
    grads = [dict() for _ in shards]

    # FFN block
    d_ln2 = []
    for r, (p, c) in enumerate(zip(shards, cache["ranks"])):
        dg = dy @ p["w2"]
        du = dg * gelu_grad(c["u"])
        grads[r]["w2"] = _tok_outer(dy, c["g"])
        grads[r]["w1"] = _tok_outer(du, cache["ln2"])
        grads[r]["b1"] = du.sum(axis=tok)
        d_ln2.append(du @ p["w1"])
        c["du"] = du
    dz2, dg2, dbeta2 = layer_norm_backward(sum(d_ln2), cache["xhat2"], cache["rstd2"], p0["ln2_g"])
    dx1 = dy + dz2

    # attention block
    d_ln1 = []
    for r, (p, c) in enumerate(zip(shards, cache["ranks"])):
        dO = (dx1 @ p["w_o"]).reshape(c["q"].shape)
        dq, dk, dv = causal_attention_backward(dO, c["q"], c["k"], c["v"], c["P"])
        b, s = dx1.shape[:2]
        dqkv = np.concatenate([dq.reshape(b, s, -1), dk.reshape(b, s, -1), dv.reshape(b, s, -1)], axis=-1)
        grads[r]["w_o"] = _tok_outer(dx1, c["O"])
        grads[r]["w_qkv"] = _tok_outer(dqkv, cache["ln1"])
        grads[r]["b_qkv"] = dqkv.sum(axis=tok)
        d_ln1.append(dqkv @ p["w_qkv"])
        c["dqkv"] = dqkv
    dz1, dg1, dbeta1 = layer_norm_backward(sum(d_ln1), cache["xhat1"], cache["rstd1"], p0["ln1_g"])
    dx = dx1 + dz1

    replicated = dict(ln1_g=dg1, ln1_b=dbeta1, ln2_g=dg2, ln2_b=dbeta2,
                      b_o=dx1.sum(axis=tok), b2=dy.sum(axis=tok))
    for g in grads:
        g.update({k: v.copy() for k, v in replicated.items()})
    return dx, grads, dict(d_ln1=d_ln1, d_ln2=d_ln2, dx1=dx1)


# --------------------------------------------------------------------------
# Stage = L blocks chained
# --------------------------------------------------------------------------

def stage_forward(x, blocks: List[Sequence[Dict[str, np.ndarray]]], n_heads_local: int, eps: float):
    """blocks[l] is the list of rank shards of block l.  Returns (y, caches)."""
    caches = []
    h = x
    for shards in blocks:
        h, c = block_forward(h, shards, n_heads_local, eps)
        caches.append(c)
    return h, caches


def stage_backward(dy, caches, blocks):
    """Returns (dx, grads[l][r], bwd[l])."""
    grads = [None] * len(blocks)
    bwd = [None] * len(blocks)
    g = dy
    for l in range(len(blocks) - 1, -1, -1):
        g, grads[l], bwd[l] = block_backward(g, caches[l], blocks[l])
    return g, grads, bwd


def shard_run(x, dy, local_blocks: List[Dict[str, np.ndarray]], n_heads_local: int, eps: float):
    """The one-GPU shard as the HIP library computes it: R = identity.  Returns a dict
    with y, dx, the forward partials p_o/p_f and backward partials d_ln1/d_ln2 per
    block, and the gradients per block."""
    blocks = [[p] for p in local_blocks]
    y, caches = stage_forward(x, blocks, n_heads_local, eps)
    dx, grads, bwd = stage_backward(dy, caches, blocks)
    return dict(
        y=y, dx=dx,
        p_o=[c["p_o"][0] for c in caches], p_f=[c["p_f"][0] for c in caches],
        d_ln1=[b["d_ln1"][0] for b in bwd], d_ln2=[b["d_ln2"][0] for b in bwd],
        grads=[g[0] for g in grads],
    )


# --------------------------------------------------------------------------
# Megatron shard map (Sec. 2 "Tensor model parallelism")
# --------------------------------------------------------------------------

def shard_block(full: Dict[str, np.ndarray], rank: int, t: int, n_heads: int) -> Dict[str, np.ndarray]:
    """Cut rank ``rank``'s slice out of a full (t = 1) block.  Rank r owns heads
    [r a/t, (r+1) a/t): its QKV rows are [its q rows; its k rows; its v rows]
    (column parallel) and its W_o columns are those heads' channels (row
    parallel); it owns FFN units [r f/t, (r+1) f/t): W1 rows and b1 (column
    parallel), W2 columns (row parallel).  LayerNorms, b_o and b2 are replicated."""
    h = full["w_o"].shape[0]
    f = full["w1"].shape[0]
    hl, fl = h // t, f // t
    c0, c1 = rank * hl, (rank + 1) * hl
    f0, f1 = rank * fl, (rank + 1) * fl
    out = {k: full[k].copy() for k in ("ln1_g", "ln1_b", "b_o", "ln2_g", "ln2_b", "b2")}
    out["w_qkv"] = np.concatenate([full["w_qkv"][part * h + c0: part * h + c1] for part in range(3)], axis=0)
    out["b_qkv"] = np.concatenate([full["b_qkv"][part * h + c0: part * h + c1] for part in range(3)], axis=0)
    out["w_o"] = full["w_o"][:, c0:c1].copy()
    out["w1"] = full["w1"][f0:f1].copy()
    out["b1"] = full["b1"][f0:f1].copy()
    out["w2"] = full["w2"][:, f0:f1].copy()
    return out


def zero_pad_block(local: Dict[str, np.ndarray], rank: int, t: int) -> Dict[str, np.ndarray]:
    """Embed rank ``rank``'s shard into a full-size block whose other ranks'
    column-parallel weights and biases (and the matching row-parallel columns) are
    zero: the one-GPU identity reduction equals this full model exactly."""
    h = local["w_o"].shape[0]
    hl = local["w_o"].shape[1]
    fl = local["w1"].shape[0]
    f = fl * t
    c0, f0 = rank * hl, rank * fl
    full = {k: local[k].copy() for k in ("ln1_g", "ln1_b", "b_o", "ln2_g", "ln2_b", "b2")}
    w_qkv = np.zeros((3 * h, h))
    b_qkv = np.zeros(3 * h)
    for part in range(3):
        w_qkv[part * h + c0: part * h + c0 + hl] = local["w_qkv"][part * hl:(part + 1) * hl]
        b_qkv[part * h + c0: part * h + c0 + hl] = local["b_qkv"][part * hl:(part + 1) * hl]
    w_o = np.zeros((h, h)); w_o[:, c0:c0 + hl] = local["w_o"]
    w1 = np.zeros((f, h)); w1[f0:f0 + fl] = local["w1"]
    b1 = np.zeros(f); b1[f0:f0 + fl] = local["b1"]
    w2 = np.zeros((h, f)); w2[:, f0:f0 + fl] = local["w2"]
    full.update(w_qkv=w_qkv, b_qkv=b_qkv, w_o=w_o, w1=w1, b1=b1, w2=w2)
    return full
