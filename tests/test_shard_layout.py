"""The shard cut used by the GPU reassembly test (the layout the C header
documents) is the oracle's Megatron shard map, which pin P4 checks on the CPU."""
import numpy as np

import oracle
from paper_2206_04959_amd import synth
from tests.test_gpu_tp_reassembly import CASES, cut


def test_documented_cut_equals_oracle_shard_map():
    for shape in CASES.values():
        full = {k: v.f64 for k, v in synth.full_block_params(shape, 0).items()}
        for r in range(shape.tp_degree):
            a = cut(full, r, shape.tp_degree)
            b = oracle.shard_block(full, r, shape.tp_degree, shape.n_heads)
            assert a.keys() == b.keys()
            for k in a:
                assert np.array_equal(a[k], b[k]), (shape.name, r, k)
