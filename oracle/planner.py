"""Plain oracle of the stage-aware recomputation planner.

TEST INFRASTRUCTURE ONLY (like the rest of this package): used by the tests,
never by the library.  It shares no code with the C implementation.

Stage-aware recomputation (Sec. 5.2): stage i of s keeps the activations of a
share alpha_i of its modules (the rest are recomputed).  Keeping them costs
(s - i) * alpha_i * M_a extra memory on top of the runtime memory M_r, because
stage i holds (s - i) micro-batches in flight.  The paper asks every stage to
use the same memory, M_r + (s - i) alpha_i M_a = M_r + (s - j) alpha_j M_a,
which fixes every alpha_i from alpha_1; shares are capped at 1; with the
shifted critical path schedule (Sec. 5.1) the penultimate stage takes the share
of the stage before it and the last stage recomputes nothing.  alpha_1 itself
is raised step by step until memory runs out (the paper catches the OOM error;
here a memory model stands in for it).

Reading taken where the paper is silent: the share alpha_i of a stage with L
blocks keeps floor(alpha_i * L) blocks (rounding down keeps the memory bound),
and the blocks that are recomputed are the first L - floor(alpha_i * L) ones.
"""
from __future__ import annotations

import math


def stage_alphas(s: int, alpha1: float):
    """[alpha_1, ..., alpha_s] (stages numbered from 1), Sec. 5.2."""
    if s < 1:
        raise ValueError("need at least one stage")
    alphas = []
    for i in range(1, s + 1):
        if i == s:
            a = 1.0
        elif i == 1:
            a = alpha1
        elif i < s - 1:
            a = min(1.0, (s - 1) * alpha1 / (s - i))
        else:  # i == s - 1
            a = alphas[-1]  # the share of stage s - 2
        alphas.append(a)
    return alphas


def stage_memory(s: int, alphas, mem_runtime: float, mem_activation: float):
    """Memory of each stage: M_r + (s - i) * alpha_i * M_a."""
    return [mem_runtime + (s - i) * a * mem_activation for i, a in enumerate(alphas, start=1)]


def largest_alpha1(s: int, mem_runtime: float, mem_activation: float, capacity: float, step: float):
    """Raise alpha_1 by `step` from 0 while every stage's memory fits."""
    best = None
    k = 0
    while k * step <= 1.0 + 1e-12:
        a1 = min(1.0, k * step)
        if max(stage_memory(s, stage_alphas(s, a1), mem_runtime, mem_activation)) <= capacity:
            best = a1
        else:
            break
        k += 1
    return best  # None: even alpha_1 = 0 does not fit


def recompute_mask(alpha: float, blocks: int) -> int:
    """Bit l set = block l of the stage is recomputed."""
    keep = math.floor(alpha * blocks + 1e-12)
    n_rc = blocks - keep
    return (1 << n_rc) - 1
