"""The work counts behind the benchmark's TFLOP/s figures (host only).

The per-block forward count is rebuilt here from the layer list (four shard
GEMMs, causal attention counted pair by pair), and the step counts from their
definitions: the backward costs twice the forward, and the recomputation of a
masked block repeats its forward without the FC2 GEMM."""
from paper_2206_04959_amd import flops, synth


def _block_forward_by_layers(s):
    T, h, hl, fl = s.tokens, s.hidden, s.local_hidden, s.local_ffn
    gemms = [(T, 3 * hl, h), (T, h, hl), (T, fl, h), (T, h, fl)]  # (M, N, K): QKV, projection, FC1, FC2
    total = sum(2 * m * n * k for m, n, k in gemms)
    d = s.head_dim
    pairs = sum(i + 1 for i in range(s.seq_len))  # causal (query, key) pairs of one sequence
    total += s.micro_batch * s.local_heads * pairs * (2 * d + 2 * d)  # q.k and p.v per pair
    return total


def test_block_forward_count_matches_the_layer_list():
    for name in ("tiny", "gpt-1.5b-stage", "gpt-2.5b-tp2", "gpt-8.3b-tp4", "gpt-20b-tp8"):
        s = synth.PRESETS[name]
        assert flops.block_forward_flops(s) == _block_forward_by_layers(s), name


def test_step_counts():
    s = synth.PRESETS["gpt-8.3b-tp4"]
    F = _block_forward_by_layers(s)
    fc2 = 2 * s.tokens * s.local_ffn * s.hidden
    R = bin(s.recompute_mask).count("1")
    assert R == 3
    assert flops.model_flops(s) == 3 * s.n_blocks * F
    assert flops.executed_flops(s) == 3 * s.n_blocks * F + R * (F - fc2)
    # the figures quoted for the 8.3B-shaped shard
    assert F == 476_753_952_768
    assert round(flops.executed_flops(s) / 1e12, 3) == 9.548
    assert round(flops.model_flops(s) / 1e12, 3) == 8.582


def test_roofline_launch_count():
    s = synth.PRESETS["gpt-8.3b-tp4"]
    # the grouped FC1/FC2 weight-gradient launch: dW2 = dy^T g and dW1 = du^T ln2
    assert flops.dw_ffn_flops(s) == 2 * (2 * s.tokens * s.local_ffn * s.hidden)
    assert round(flops.dw_ffn_flops(s) / 1e9, 1) == 309.2
