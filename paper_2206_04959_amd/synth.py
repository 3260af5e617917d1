"""Seeded synthetic workloads for one GPU's share of a GPT pipeline stage.

This module is shared by the HIP path's tests/benchmark and by the fp64
oracle's tests.  It holds shapes and random numbers only: no step of the
forward or backward pass is computed here.

Shapes follow the GPT model family the paper evaluates (Sec. 6.1 "Models and
Datasets": GPT-like decoder models, sequence length 1024) at the widths of the
1.5B/2.5B/8.3B/20B configurations used for measurement, each cut to one
pipeline stage and one tensor-model-parallel rank (Sec. 2 "Tensor model
parallelism", Sec. 5.3).  The paper trains on OpenWebText; per-GPU stage compute
depends only on shapes, so seeded N(0, 1) hidden states of the same shape stand
in for the embedded tokens.

Value recipe (the paper states none):
  * weights W ~ N(0, 0.02); biases ~ N(0, 0.02); LayerNorm gamma = 1 + N(0, 0.02),
    beta ~ N(0, 0.02);
  * stage input x ~ N(0, x_std) (0.02 for the tiny check case, 1.0 otherwise);
  * upstream gradient dy ~ N(0, 1).
In bf16 mode every value is drawn in fp32 and rounded to the nearest bf16
(ties to even); both the GPU path and the oracle receive exactly those values.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List

import numpy as np

# Per-block parameter tensors, in the order the flat parameter buffer stores them.
PARAM_NAMES = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
               "ln2_g", "ln2_b", "w1", "b1", "w2", "b2")


@dataclasses.dataclass(frozen=True)
class StageShape:
    """Global (t = 1) model dimensions plus the shard/schedule knobs."""
    name: str
    n_blocks: int          # L: consecutive transformer blocks in the stage
    hidden: int            # h
    n_heads: int           # a
    ffn: int               # f
    seq_len: int           # s
    micro_batch: int       # b
    tp_degree: int = 1     # t
    n_sub: int = 1         # n: sub-micro-batches per micro-batch
    recompute_mask: int = 0  # bit l set: block l keeps only its input
    dtype: str = "bf16"    # "bf16" (fp32 accumulate) or "fp32" check mode
    x_std: float = 1.0
    w_std: float = 0.02
    ln_eps: float = 1e-5
    seed: int = 2206

    # --- derived sizes -------------------------------------------------
    @property
    def head_dim(self) -> int:
        return self.hidden // self.n_heads

    @property
    def local_heads(self) -> int:
        return self.n_heads // self.tp_degree

    @property
    def local_hidden(self) -> int:
        return self.hidden // self.tp_degree

    @property
    def local_ffn(self) -> int:
        return self.ffn // self.tp_degree

    @property
    def tokens(self) -> int:
        return self.micro_batch * self.seq_len

    def replace(self, **kw) -> "StageShape":
        return dataclasses.replace(self, **kw)

    def local_param_shapes(self) -> Dict[str, tuple]:
        h, hl, fl = self.hidden, self.local_hidden, self.local_ffn
        return {
            "ln1_g": (h,), "ln1_b": (h,),
            "w_qkv": (3 * hl, h), "b_qkv": (3 * hl,),
            "w_o": (h, hl), "b_o": (h,),
            "ln2_g": (h,), "ln2_b": (h,),
            "w1": (fl, h), "b1": (fl,),
            "w2": (h, fl), "b2": (h,),
        }


# The workloads: a tiny fp32 check case and four stage shards.
TINY = StageShape("tiny", n_blocks=1, hidden=256, n_heads=4, ffn=1024, seq_len=128,
                  micro_batch=2, tp_degree=1, n_sub=1, recompute_mask=0,
                  dtype="fp32", x_std=0.02, seed=2206)
GPT_1_5B = StageShape("gpt-1.5b-stage", n_blocks=12, hidden=1600, n_heads=25, ffn=6400,
                      seq_len=1024, micro_batch=4, tp_degree=1, n_sub=2, seed=2207)
GPT_2_5B = StageShape("gpt-2.5b-tp2", n_blocks=8, hidden=1920, n_heads=20, ffn=7680,
                      seq_len=1024, micro_batch=4, tp_degree=2, n_sub=2, seed=2208)
GPT_8_3B = StageShape("gpt-8.3b-tp4", n_blocks=6, hidden=3072, n_heads=32, ffn=12288,
                      seq_len=1024, micro_batch=8, tp_degree=4, n_sub=4,
                      recompute_mask=0b000111, seed=2209)
GPT_20B = StageShape("gpt-20b-tp8", n_blocks=4, hidden=6144, n_heads=48, ffn=24576,
                     seq_len=2048, micro_batch=4, tp_degree=8, n_sub=4,
                     recompute_mask=0b1111, seed=2210)

PRESETS = {s.name: s for s in (TINY, GPT_1_5B, GPT_2_5B, GPT_8_3B, GPT_20B)}


# --- bf16 rounding (input preparation only) ---------------------------------

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest, ties to even."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


class Tensor:
    """One synthetic tensor: fp64 values (exactly what the device receives) and
    the device-format payload (bf16 bits as uint16, or fp32)."""

    def __init__(self, f64: np.ndarray, payload: np.ndarray):
        self.f64 = f64
        self.payload = payload

    @property
    def shape(self):
        return self.f64.shape


def _draw(rng: np.random.Generator, shape, mean: float, std: float, dtype: str) -> Tensor:
    v = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(std) + np.float32(mean)
    if dtype == "bf16":
        bits = f32_to_bf16_bits(v)
        return Tensor(bf16_bits_to_f64(bits), bits)
    if dtype == "fp32":
        return Tensor(v.astype(np.float64), v)
    raise ValueError(f"unknown dtype {dtype!r}")


def _rng(shape: StageShape, *key: int) -> np.random.Generator:
    # Independent, order-free streams: one per (seed, tensor kind, block, rank).
    return np.random.default_rng([shape.seed, *key])


_KIND = {name: i for i, name in enumerate(PARAM_NAMES)}
_KIND_X, _KIND_DY = 100, 101


def _param_dist(name: str, std: float):
    if name in ("ln1_g", "ln2_g"):
        return 1.0, std
    return 0.0, std


def full_block_params(shape: StageShape, block: int) -> Dict[str, Tensor]:
    """Parameters of the whole (t = 1) block ``block``; see ``shard`` helpers in the
    oracle for how a rank's slice is cut from these."""
    full = shape.replace(tp_degree=1)
    out = {}
    for name, shp in full.local_param_shapes().items():
        mean, std = _param_dist(name, shape.w_std)
        out[name] = _draw(_rng(shape, 1000 + _KIND[name], block), shp, mean, std, shape.dtype)
    return out


def local_block_params(shape: StageShape, block: int, rank: int = 0) -> Dict[str, Tensor]:
    """Parameters of tensor-parallel rank ``rank``'s shard of block ``block``, drawn
    directly at the shard's shape (same distribution as a slice of a full draw)."""
    out = {}
    for name, shp in shape.local_param_shapes().items():
        mean, std = _param_dist(name, shape.w_std)
        out[name] = _draw(_rng(shape, _KIND[name], block, rank), shp, mean, std, shape.dtype)
    return out


def stage_params(shape: StageShape, rank: int = 0) -> List[Dict[str, Tensor]]:
    return [local_block_params(shape, l, rank) for l in range(shape.n_blocks)]


def stage_input(shape: StageShape) -> Tensor:
    """x: [micro_batch, seq_len, hidden]."""
    return _draw(_rng(shape, _KIND_X), (shape.micro_batch, shape.seq_len, shape.hidden),
                 0.0, shape.x_std, shape.dtype)


def upstream_grad(shape: StageShape) -> Tensor:
    """dy: [micro_batch, seq_len, hidden] ~ N(0, 1)."""
    return _draw(_rng(shape, _KIND_DY), (shape.micro_batch, shape.seq_len, shape.hidden),
                 0.0, 1.0, shape.dtype)
