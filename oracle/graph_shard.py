"""Plain oracle of the graph-sharding algorithm (Sec. 4.2, Alg. 1 and Alg. 2).

TEST INFRASTRUCTURE ONLY (like the rest of this package): used by the tests,
never by the library.  It shares no code with the C implementation.

The model graph is a DAG whose nodes are visited in topological order.  Each
node is placed in a subgraph next to its farthest dependency (Alg. 1); a
subgraph is closed once the parameters it holds exceed sum(params) / k, and its
output is the node that closed it plus every visited "common" node that still
has users (Alg. 2).  The result is a sequence of subgraphs that can run one
after the other, each taking the previous one's outputs and the graph inputs
it is the first to use.

Notation follows the paper: C common node -> remaining user count, X graph
inputs, I graph input -> first user, M node -> subgraph id, S_outs subgraph id
-> outputs, N visited nodes, D node -> parameter count, p the threshold.

Readings where the listings are silent or ambiguous:
  * graph inputs are not visited as nodes: they are the set X; a node that
    reads the same graph input twice is its first user, not a dependency of
    itself;
  * when a node's farthest dependency lies in an older subgraph, the nodes
    visited after that dependency move into its subgraph.  The dependency node
    itself keeps its subgraph: the listing assigns it too, which only matters
    when the dependency is the output of an earlier subgraph and would move an
    output out of the subgraph that produces it;
  * reopening subgraph s by such a merge discards the outputs recorded for s
    and every later subgraph: those subgraphs no longer exist, and s records
    its outputs again when it closes;
  * the last subgraph is emitted even if it never exceeded the threshold, and
    its outputs are the graph outputs;
  * a subgraph's inputs are the previous subgraph's outputs plus the graph
    inputs whose first user it holds (in graph-input order);
  * the outputs recorded when a subgraph closes list the common nodes in visit
    order, then the closing node.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple


def search_dependency(n, args, s, C, X, I, M, S_outs, N):
    """Alg. 1: the smallest subgraph id node n may join and the node that
    forces it (None if n may stay in subgraph s)."""
    s_min, n_min = s, None
    outputs = {o for outs in S_outs.values() for o in outs}
    for arg in args:
        if arg in C:  # a common node: no dependency, one user fewer
            C[arg] -= 1
        elif arg in X:  # a graph input: stay with its first user
            if I.get(arg) is None:
                I[arg] = n
            elif I[arg] != n and M[I[arg]] < s_min:  # (n reading it twice is no dependency)
                s_min, n_min = M[I[arg]], I[arg]
        elif arg in outputs:  # an output of a previous subgraph
            if M[arg] + 1 < s_min:
                s_min, n_min = M[arg] + 1, arg
        elif arg in M and arg != N[-1]:  # another visited node, not the last one
            if M[arg] < s_min:
                s_min, n_min = M[arg], arg
    return s_min, n_min


def graph_shard(nodes: Sequence[Tuple[str, Sequence[str]]], X: Sequence[str], graph_outputs: Sequence[str],
                k: int, D: Dict[str, int], C: Dict[str, int]):
    """Alg. 2.  nodes: (name, argument names) in topological order, graph
    inputs excluded.  Returns (M, subgraphs) with subgraphs a list of dicts
    {"nodes", "inputs", "outputs"} in execution order."""
    C = dict(C)
    X_order = list(X)
    X = set(X)
    M: Dict[str, int] = {}
    I: Dict[str, str] = {}
    S_outs: Dict[int, List[str]] = {}
    N: List[str] = []
    p = sum(D.values()) / k
    s = 0
    for n, args in nodes:
        s_min, n_min = search_dependency(n, args, s, C, X, I, M, S_outs, N)
        if s_min < s:
            s = s_min
            for n_prev in reversed(N):  # nodes after n_min join its subgraph
                if n_prev == n_min:
                    break
                M[n_prev] = s_min
            for t in [t for t in S_outs if t >= s_min]:  # subgraph s_min is open again
                del S_outs[t]
        M[n] = s
        N.append(n)
        p_s = sum(D.get(m, 0) for m in M if M[m] == s)
        if p_s > p:
            S_outs[s] = [n_c for n_c in C if n_c in M and C[n_c] > 0]
            S_outs[s].append(n)
            s += 1
    last = max(M.values()) if M else -1
    subgraphs = []
    for s_i in range(last + 1):
        g_nodes = [n for n, _ in nodes if M[n] == s_i]
        g_inputs = list(S_outs.get(s_i - 1, [])) + [x for x in X_order if I.get(x) in g_nodes]
        g_outputs = list(S_outs[s_i]) if s_i < last else list(graph_outputs)
        subgraphs.append({"nodes": g_nodes, "inputs": g_inputs, "outputs": g_outputs})
    return M, subgraphs


def from_fx(gm, common_min_users: int = 2):
    """The algorithm's inputs from a torch.fx GraphModule: visited nodes with
    their argument nodes, graph inputs X (placeholders), graph outputs, D (the
    parameter count of each called module) and C (common nodes: nodes that no
    parameter-carrying node feeds, directly or through other nodes, and that
    are used at least `common_min_users` times, with their use counts)."""
    import torch.fx as fx

    X, nodes, outs, D = [], [], [], {}
    fed_by_params = set()
    users: Dict[str, int] = {}
    for node in gm.graph.nodes:
        if node.op == "placeholder":
            X.append(node.name)
            continue
        if node.op == "output":
            outs = [a.name for a in node.all_input_nodes]
            continue
        # one entry per use of a node among the arguments (Alg. 1 walks n.args)
        args = []
        fx.node.map_arg((node.args, node.kwargs), lambda a: args.append(a.name))
        nodes.append((node.name, args))
        for a in args:
            users[a] = users.get(a, 0) + 1
        params = 0
        if node.op == "call_module":
            params = sum(t.numel() for t in gm.get_submodule(node.target).parameters())
        elif node.op == "get_attr":
            params = getattr(gm, node.target).numel() if hasattr(getattr(gm, node.target), "numel") else 0
        D[node.name] = params
        if params > 0 or any(a in fed_by_params for a in args):
            fed_by_params.add(node.name)
    C = {n: users.get(n, 0) for n, _ in nodes
         if n not in fed_by_params and users.get(n, 0) >= common_min_users}
    return nodes, X, outs, D, C
