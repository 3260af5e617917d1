"""Algorithmic work of one stage step (counted as the method must compute it).

Per block forward, one rank's shard, T = b*s tokens:
  GEMMs      2*T*h*(3h/t) + 2*T*(h/t)*h + 2*T*h*(f/t) + 2*T*(f/t)*h
  attention  2*b*(h/t)*s*(s+1)   (causal: Q K^T and P V over the lower triangle
                                  including the diagonal)
The backward pass costs twice the forward (Sec. 5.1 of the paper takes the same
ratio), and each recomputed block repeats its forward once, except the FC2 GEMM:
its output is the next block's (checkpointed) input, and the backward needs
only FC2's input, so the recomputation leaves it out.  Tile padding and the
attention backward's rebuilding of P are not counted.
"""
from __future__ import annotations

from .synth import StageShape


def block_forward_flops(s: StageShape) -> float:
    T, h, hl, fl = s.tokens, s.hidden, s.local_hidden, s.local_ffn
    gemm = 2.0 * T * h * (3 * hl) + 2.0 * T * hl * h + 2.0 * T * h * fl + 2.0 * T * fl * h
    attn = 2.0 * s.micro_batch * hl * s.seq_len * (s.seq_len + 1)
    return gemm + attn


def recomputed_blocks(s: StageShape) -> int:
    return bin(s.recompute_mask).count("1")


def fc2_forward_flops(s: StageShape) -> float:
    return 2.0 * s.tokens * s.local_ffn * s.hidden


def executed_flops(s: StageShape) -> float:
    """Forward + recompute (all but FC2) + backward of the whole stage for one
    micro-batch."""
    return 3 * s.n_blocks * block_forward_flops(s) + recomputed_blocks(s) * (block_forward_flops(s)
                                                                             - fc2_forward_flops(s))


def model_flops(s: StageShape) -> float:
    """Forward + backward only (what the stage would cost without recomputation)."""
    return 3 * s.n_blocks * block_forward_flops(s)


def dw_gemm_flops(s: StageShape) -> float:
    """All weight-gradient GEMMs of one block (= the block's forward GEMM work)."""
    T, h, hl, fl = s.tokens, s.hidden, s.local_hidden, s.local_ffn
    return 2.0 * T * (3 * hl * h + h * hl + fl * h + h * fl)


def dw_ffn_flops(s: StageShape) -> float:
    """The grouped weight-gradient GEMM of FC1 and FC2 of one block (one launch)."""
    T, h, fl = s.tokens, s.hidden, s.local_ffn
    return 2.0 * T * (fl * h + h * fl)
