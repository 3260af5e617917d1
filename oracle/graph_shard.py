"""Plain oracle of the graph-sharding algorithm (Sec. 4.2).

TEST INFRASTRUCTURE ONLY (like the rest of this package): used by the tests,
never by the library.  It shares no code with the C implementation.

What the section states, and what this oracle computes:
  * the model graph is a DAG; its nodes are visited once, in topological order,
    while subgraph ids are handed out from 0;
  * a node must share a subgraph with its farthest dependency.  Its arguments
    can tie it to: a graph input (the node goes where that input's first reader
    went), an output of an earlier subgraph (the node may sit in the subgraph
    right after its producer), or any other node visited before it except the
    one visited just before (the node goes where that node is).  Common nodes
    (nodes used by many blocks, such as the attention mask) tie nothing; their
    remaining uses are counted down instead;
  * when that dependency lies in an earlier subgraph than the current one, the
    current subgraph becomes that one, and every node visited after the
    dependency moves into it;
  * a subgraph closes as soon as the parameters of its nodes exceed the total
    over the number of subgraphs asked for; what it hands on is every visited
    common node that still has uses, then the node that closed it;
  * each subgraph's inputs are what the one before it handed on, plus the graph
    inputs it reads first, so the subgraphs run one after the other.

Readings where the section is silent or ambiguous:
  * graph inputs are not visited as nodes; a node that reads the same graph
    input twice is its first reader, not a dependency of itself;
  * the dependency node itself keeps its subgraph when later nodes move into
    its subgraph (moving it would take an output out of the subgraph that
    produces it);
  * moving nodes back into subgraph s reopens s: the outputs recorded for s and
    every later subgraph are dropped, and s records its outputs again when it
    closes;
  * the last subgraph is emitted even if it never reached the threshold, and
    its outputs are the graph outputs;
  * the graph inputs of a subgraph are listed in graph-input order, its handed-
    on common nodes in visit order, then the closing node.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple


class _Walk:
    """State of one pass over the graph."""

    def __init__(self, graph_inputs: Sequence[str], params: Dict[str, int], common: Dict[str, int], k: int):
        self.graph_inputs = set(graph_inputs)
        self.params = params
        self.uses_left = dict(common)          # common node -> uses not yet visited
        self.first_reader: Dict[str, str] = {}  # graph input -> first node reading it
        self.place: Dict[str, int] = {}        # visited node -> subgraph id
        self.order: List[str] = []             # visited nodes, in visit order
        self.handed_on: Dict[int, List[str]] = {}  # closed subgraph -> what it hands on
        self.limit = sum(params.values()) / k
        self.current = 0

    def _tie(self, node: str, arg: str) -> Optional[Tuple[int, str]]:
        """(subgraph the argument ties `node` to, the node responsible), or None."""
        if arg in self.uses_left:
            self.uses_left[arg] -= 1
            return None
        if arg in self.graph_inputs:
            reader = self.first_reader.setdefault(arg, node)
            return None if reader == node else (self.place[reader], reader)
        if any(arg in outs for outs in self.handed_on.values()):
            return self.place[arg] + 1, arg
        if arg in self.place and arg != self.order[-1]:
            return self.place[arg], arg
        return None

    def farthest_dependency(self, node: str, args: Sequence[str]) -> Tuple[int, Optional[str]]:
        best, anchor = self.current, None
        for arg in args:
            t = self._tie(node, arg)
            if t is not None and t[0] < best:
                best, anchor = t
        return best, anchor

    def pull_back(self, target: int, anchor: str) -> None:
        """Nodes visited after `anchor` join subgraph `target`, which reopens."""
        for name in self.order[self.order.index(anchor) + 1:]:
            self.place[name] = target
        for sub in [t for t in self.handed_on if t >= target]:
            del self.handed_on[sub]
        self.current = target

    def visit(self, node: str, args: Sequence[str]) -> None:
        target, anchor = self.farthest_dependency(node, args)
        if target < self.current:
            self.pull_back(target, anchor)
        self.place[node] = self.current
        self.order.append(node)
        held = sum(self.params.get(m, 0) for m, sub in self.place.items() if sub == self.current)
        if held > self.limit:
            live_common = [c for c in self.uses_left if c in self.place and self.uses_left[c] > 0]
            self.handed_on[self.current] = live_common + [node]
            self.current += 1


def graph_shard(nodes: Sequence[Tuple[str, Sequence[str]]], X: Sequence[str], graph_outputs: Sequence[str],
                k: int, D: Dict[str, int], C: Dict[str, int]):
    """nodes: (name, argument names) in topological order, graph inputs
    excluded; X: graph inputs; D: parameters per node; C: common nodes with
    their use counts; k: subgraphs asked for.  Returns (node -> subgraph id,
    subgraphs), the subgraphs a list of dicts {"nodes", "inputs", "outputs"} in
    execution order."""
    walk = _Walk(X, D, C, k)
    for name, args in nodes:
        walk.visit(name, args)
    n_sub = max(walk.place.values()) + 1 if walk.place else 0
    subgraphs = []
    for sub in range(n_sub):
        members = [name for name, _ in nodes if walk.place[name] == sub]
        reads_first = [x for x in X if walk.first_reader.get(x) in members]
        subgraphs.append({
            "nodes": members,
            "inputs": list(walk.handed_on.get(sub - 1, [])) + reads_first,
            "outputs": list(walk.handed_on[sub]) if sub < n_sub - 1 else list(graph_outputs),
        })
    return dict(walk.place), subgraphs


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
