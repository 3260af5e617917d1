"""Graph sharding of a torch.fx model graph (paper Sec. 4.2) through the C ABI.

    subgraphs = shard_fx(gm, k)

The algorithm itself (Alg. 1 + Alg. 2) runs in the HIP library's host code
(`merak_graph_shard`); this module turns a GraphModule into the node arrays
that call takes and builds one GraphModule per subgraph from the result.  The
subgraphs run in sequence: subgraph j takes the previous one's outputs and the
graph inputs it is the first to use, in that order, and returns its outputs as
a tuple (the last one returns what the whole graph returns).

What a node contributes:
  * parameters: the parameter count of the module a `call_module` node calls
    (other nodes hold none);
  * common nodes: values that no parameter-carrying node feeds, directly or
    through other nodes, and that are used at least twice (position ids, a
    causal mask ...).  The algorithm lets every subgraph read them.
"""
from __future__ import annotations

import ctypes
from typing import List

import numpy as np

from . import binding as B

NODE_COMPUTE, NODE_INPUT, NODE_COMMON = 0, 1, 2


def graph_arrays(gm):
    """(nodes, kind, params, arg_ptr, arg_idx, common_uses, outputs) of a
    GraphModule, nodes in graph order without the output node."""
    import torch.fx as fx

    nodes = [n for n in gm.graph.nodes if n.op != "output"]
    out_node = next(n for n in gm.graph.nodes if n.op == "output")
    index = {n: i for i, n in enumerate(nodes)}
    kind = np.zeros(len(nodes), dtype=np.int32)
    params = np.zeros(len(nodes), dtype=np.int64)
    arg_ptr = np.zeros(len(nodes) + 1, dtype=np.int32)
    args: List[int] = []
    param_fed = np.zeros(len(nodes), dtype=bool)
    for i, n in enumerate(nodes):
        uses: List[int] = []
        fx.node.map_arg((n.args, n.kwargs), lambda a: uses.append(index[a]))
        args.extend(uses)
        arg_ptr[i + 1] = len(args)
        if n.op == "placeholder":
            kind[i] = NODE_INPUT
        elif n.op == "call_module":
            params[i] = sum(p.numel() for p in gm.get_submodule(n.target).parameters())
        param_fed[i] = params[i] > 0 or any(param_fed[a] for a in uses)
    arg_idx = np.asarray(args, dtype=np.int32)
    common_uses = np.bincount(arg_idx, minlength=len(nodes)).astype(np.int32)
    for i, n in enumerate(nodes):
        if kind[i] != NODE_INPUT and not param_fed[i] and common_uses[i] >= 2:
            kind[i] = NODE_COMMON
    common_uses[kind != NODE_COMMON] = 0
    outputs: List[int] = []
    fx.node.map_arg(out_node.args, lambda a: outputs.append(index[a]))
    return nodes, kind, params, arg_ptr, arg_idx, common_uses, np.asarray(outputs, dtype=np.int32)


def shard_arrays(kind, params, arg_ptr, arg_idx, common_uses, outputs, k: int):
    """Run merak_graph_shard: (subgraph id per node, [(input indices, output
    indices)] per subgraph)."""
    n = len(kind)
    sub = np.zeros(n, dtype=np.int32)
    n_sub = ctypes.c_int32()
    io_ptr = np.zeros(2 * n + 1, dtype=np.int32)
    cap = max(16, 4 * n)
    P = lambda a: a.ctypes.data_as(ctypes.c_void_p)  # noqa: E731
    arg_idx = np.ascontiguousarray(arg_idx, dtype=np.int32)
    while True:
        io_idx = np.zeros(cap, dtype=np.int32)
        st = B.lib().merak_graph_shard(n, P(kind), P(params), P(arg_ptr), P(arg_idx) if len(arg_idx) else None,
                                       P(common_uses), len(outputs), P(outputs) if len(outputs) else None, int(k),
                                       P(sub), ctypes.byref(n_sub), P(io_ptr), P(io_idx), cap)
        if st == -5:  # MERAK_ERR_WORKSPACE: io_ptr[2 * n_sub] holds the size needed
            cap = int(io_ptr[2 * n_sub.value])
            continue
        B._check(st, "merak_graph_shard")
        break
    S = n_sub.value
    io = [(io_idx[io_ptr[2 * j]:io_ptr[2 * j + 1]].tolist(), io_idx[io_ptr[2 * j + 1]:io_ptr[2 * j + 2]].tolist())
          for j in range(S)]
    return sub, io


def shard_fx(gm, k: int):
    """Shard GraphModule gm into at most about k parameter-balanced subgraphs
    (Alg. 2's threshold sum(params) / k).  Returns a list of GraphModules (they
    share gm's submodules)."""
    import torch.fx as fx

    nodes, kind, params, arg_ptr, arg_idx, common_uses, outputs = graph_arrays(gm)
    sub, io = shard_arrays(kind, params, arg_ptr, arg_idx, common_uses, outputs, k)
    mods = []
    for j, (ins, outs) in enumerate(io):
        g = fx.Graph()
        env = {}
        for i in ins:
            env[nodes[i]] = g.placeholder(nodes[i].name)
        for i, n in enumerate(nodes):
            if sub[i] == j:
                env[n] = g.node_copy(n, lambda a: env[a])
        g.output(tuple(env[nodes[i]] for i in outs))
        mods.append(fx.GraphModule(gm, g))
    return mods


def run_sequence(mods, *inputs, input_names=None):
    """Run shard_fx's subgraphs one after the other on the graph inputs (in
    placeholder order) and return the last subgraph's outputs."""
    names = input_names
    values = dict(zip(names, inputs)) if names else {}
    carry = ()
    for m in mods:
        ph = [n.name for n in m.graph.nodes if n.op == "placeholder"]
        n_carry = len(carry)
        args = list(carry) + [values[p] for p in ph[n_carry:]]
        carry = m(*args)
    return carry
