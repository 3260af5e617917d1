"""Helpers shared by the oracle tests: fp64 parameter dicts from the seeded generator."""
import numpy as np

from paper_2206_04959_amd import synth


def f64_params(tensors):
    return {k: v.f64 for k, v in tensors.items()}


def local_stage(shape, rank=0):
    return [f64_params(synth.local_block_params(shape, l, rank)) for l in range(shape.n_blocks)]


def full_stage(shape):
    return [f64_params(synth.full_block_params(shape, l)) for l in range(shape.n_blocks)]


def rel_max_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    denom = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / (denom if denom > 0 else 1.0))
