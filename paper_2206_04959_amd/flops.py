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


def gemm_forward_flops(s: StageShape) -> float:
    """The four shard GEMMs of one block's forward pass."""
    T, h, hl, fl = s.tokens, s.hidden, s.local_hidden, s.local_ffn
    return 2.0 * T * h * (3 * hl) + 2.0 * T * hl * h + 2.0 * T * h * fl + 2.0 * T * fl * h


def attention_forward_flops(s: StageShape) -> float:
    return 2.0 * s.micro_batch * s.local_hidden * s.seq_len * (s.seq_len + 1)


def dw_attn_flops(s: StageShape) -> float:
    """The grouped weight-gradient GEMM of QKV and the projection of one block (one launch)."""
    T, h, hl = s.tokens, s.hidden, s.local_hidden
    return 2.0 * T * (3 * hl * h + h * hl)


def class_work(s: StageShape) -> dict:
    """Algorithmic work of one stage step per kernel class: {class name: (amount,
    unit, bound)}.  FLOP for the MFMA-bound classes, bytes (each input read once,
    each output written once) for the memory-bound ones.  The class names are
    the library's timing classes (merak_stage_set_timing)."""
    L, R = s.n_blocks, recomputed_blocks(s)
    T, h, hl, fl = s.tokens, s.hidden, s.local_hidden, s.local_ffn
    e = 2 if s.dtype == "bf16" else 4
    ln_fwd = 2.0 * T * h * e + 8.0 * T            # read x, write y, write mean and rstd
    ln_bwd = 4.0 * T * h * e + 8.0 * T            # read dout, x, the residual gradient; write dx; read stats
    # bias sums read dy, du, dqkv and dx1 once; LayerNorm-parameter sums read
    # each LayerNorm's output gradient and input once (plus its statistics)
    reduce = T * e * (h + fl + 3 * hl + h + 4 * h) + 2 * 8.0 * T
    return {
        "GEMM_FWD": (L * gemm_forward_flops(s) + R * (gemm_forward_flops(s) - fc2_forward_flops(s)), "FLOP", "mfma"),
        "GEMM_DX": (L * gemm_forward_flops(s), "FLOP", "mfma"),
        "GEMM_DW": (L * dw_ffn_flops(s), "FLOP", "mfma"),
        "GEMM_DW_ATTN": (L * dw_attn_flops(s), "FLOP", "mfma"),
        "ATTN_FWD": ((L + R) * attention_forward_flops(s), "FLOP", "mfma"),
        "ATTN_BWD": (2.0 * L * attention_forward_flops(s), "FLOP", "mfma"),
        "LN_FWD": (2 * (L + R) * ln_fwd, "B", "hbm"),
        "LN_BWD": (2 * L * ln_bwd, "B", "hbm"),
        "REDUCE": (L * reduce, "B", "hbm"),
    }
