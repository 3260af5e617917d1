"""Plain oracle of the pipeline schedules of Sec. 5.1 and their bubble ratios.

TEST INFRASTRUCTURE ONLY (like the rest of this package).  It shares no code
with the C implementation.

Costs (Sec. 5.1): forward T_m, recomputation T_m, backward 2 T_m per
micro-batch and stage.  Ops are ("F" | "R" | "B" | "RB", micro-batch); "RB" is
a backward that recomputes the forward itself (plain 1F1B with activation
recomputation).  Dependencies: F of stage i needs F of stage i-1 (its input);
B needs B of stage i+1 (its output gradient) and the stage's own R of that
micro-batch when there is one; R needs only the stage's stored input, i.e.
nothing from other stages (Gpipe's observation the paper builds on).

Schedules, s stages numbered 0..s-1, m micro-batches:
* 1F1B: stage i runs s-1-i forwards, then alternates one forward with one
  backward ("RB"), then the remaining backwards.  Bubble ratio (s-1)/m.
* early recomputation: the same order with R split out of the backward, so it
  runs as soon as the stage is free.  Bubble ratio 3(s-1)/(4m).
* shifted critical path (SCP): the last stage keeps its one activation and
  skips recomputation; the penultimate stage runs one forward ahead, in the
  bubble left by its first backward (its order starts F0 F1 R0 F2 B0, then
  R_j B_j F_{j+2}); the other stages as in early recomputation.  Bubble ratio
  3(s-2)/(4m).
Reading taken: the paper draws the SCP order in a figure and describes it in
one sentence; the order above is the one that reaches its stated bubble time
3(s-2) T_m (checked by simulation for many s, m).
"""
from __future__ import annotations

COST = {"F": 1.0, "R": 1.0, "B": 2.0, "RB": 3.0}


def stage_ops(kind: str, s: int, m: int, i: int):
    """Op list of stage i."""
    if kind not in ("1f1b", "early", "scp"):
        raise ValueError(kind)
    if kind == "scp" and i == s - 1:
        ops = []
        for j in range(m):
            ops += [("F", j), ("B", j)]
        return ops
    if kind == "scp" and i == s - 2 and m >= 2:
        ops = [("F", 0), ("F", 1), ("R", 0)]
        nf = 2
        if nf < m:
            ops.append(("F", nf))
            nf += 1
        ops.append(("B", 0))
        for j in range(1, m):
            ops += [("R", j), ("B", j)]
            if nf < m:
                ops.append(("F", nf))
                nf += 1
        return ops
    warm = min(s - 1 - i, m)
    ops = [("F", j) for j in range(warm)]
    nf = warm
    for j in range(m):
        if nf < m:
            ops.append(("F", nf))
            nf += 1
        if kind == "1f1b":
            ops.append(("RB", j))
        else:
            ops += [("R", j), ("B", j)]
    return ops


def simulate(kind: str, s: int, m: int, cost=COST):
    """Greedy in-order execution; returns (makespan, busy time per stage, finish time of every op)."""
    plans = [stage_ops(kind, s, m, i) for i in range(s)]
    finish = {}
    free = [0.0] * s
    pos = [0] * s
    left = sum(len(p) for p in plans)
    while left:
        moved = False
        for i in range(s):
            if pos[i] == len(plans[i]):
                continue
            op, j = plans[i][pos[i]]
            deps = []
            if op == "F" and i > 0:
                deps.append(("F", i - 1, j))
            if op in ("B", "RB"):
                if i < s - 1:
                    deps.append(("B", i + 1, j))
                if op == "B" and ("R", j) in plans[i]:
                    deps.append(("R", i, j))
            if all(d in finish for d in deps):
                start = max([free[i]] + [finish[d] for d in deps])
                free[i] = start + cost[op]
                finish[("B" if op == "RB" else op, i, j)] = free[i]
                pos[i] += 1
                left -= 1
                moved = True
        if not moved:
            raise RuntimeError("schedule deadlocks")
    busy = [sum(cost[op] for op, _ in p) for p in plans]
    return max(free), busy, finish


def bubble_ratio(kind: str, s: int, m: int) -> float:
    """(makespan - 4 m T_m) / (4 m T_m), the paper's idle-to-running ratio."""
    makespan, _, _ = simulate(kind, s, m)
    return (makespan - 4.0 * m) / (4.0 * m)
