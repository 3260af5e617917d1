"""Host-only checks of the C ABI: the library loads, exports every function the
header declares, and rejects bad configurations/arguments before touching the GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2206_04959_amd import binding as B
from paper_2206_04959_amd import synth

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "merak_stage.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+char\s*\*|int|size_t)\s+(merak_\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert len(names) >= 15
    lib = B.lib()
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B._SIGS), "binding signatures out of sync with the header"


def test_status_strings():
    lib = B.lib()
    assert lib.merak_status_str(0) == b"ok"
    assert lib.merak_status_str(-3) == b"call-order violation"
    assert lib.merak_status_str(12345) == b"unknown status"


@pytest.mark.parametrize("name", sorted(synth.PRESETS))
def test_presets_validate(name):
    assert B.validate(B.make_config(synth.PRESETS[name])) == 0


@pytest.mark.parametrize("change,status", [
    (dict(n_blocks=0), -2), (dict(n_blocks=65), -2),
    (dict(n_heads=5), -2),                      # 256 % 5 != 0
    (dict(tp_degree=3), -2),                    # heads % t
    (dict(micro_batch=3, n_sub=2), -2),         # b % n
    (dict(seq_len=100), -2),                    # seq % 64
    (dict(hidden=320, n_heads=4, ffn=1280), -7),  # head_dim 80 unsupported
    (dict(recompute_mask=0b10), -2),            # bit >= n_blocks
    (dict(ln_eps=0.0), -2),
    (dict(hidden=192, n_heads=2, ffn=768, tp_degree=2), -2),  # h/t = 96 not a multiple of 64
    # bf16: a [b*s, ffn] activation of 2^20 rows (+256 rows of tile padding) passes 2^31 bytes;
    # the fp32 check mode has no such limit
    (dict(micro_batch=8192, dtype="bf16"), -2), (dict(micro_batch=8192, dtype="fp32"), 0),
])
def test_bad_configs_rejected(change, status):
    cfg = B.make_config(synth.TINY.replace(**change))
    assert B.validate(cfg) == status


def test_bad_dtype_rejected():
    cfg = B.make_config(synth.TINY)
    cfg.dtype = 7
    assert B.validate(cfg) == -1


@pytest.mark.parametrize("name", sorted(synth.PRESETS))
def test_param_layout_is_dense_aligned_and_disjoint(name):
    shape = synth.PRESETS[name]
    cfg = B.make_config(shape)
    total, offs = B.param_layout(cfg)
    sizes = [int(np.prod(s)) for s in shape.local_param_shapes().values()]
    spans = []
    for l in range(shape.n_blocks):
        for i, n in enumerate(sizes):
            assert offs[l, i] % 64 == 0
            spans.append((offs[l, i], offs[l, i] + n))
    spans.sort()
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        assert a1 <= b0
    assert spans[-1][1] <= total < spans[-1][1] + 64 * 12


def test_workspace_sizes_follow_recompute_mask():
    base = synth.GPT_8_3B
    ws0, rc0 = B.workspace_bytes(B.make_config(base.replace(recompute_mask=0)))
    ws3, rc3 = B.workspace_bytes(B.make_config(base))
    wsa, rca = B.workspace_bytes(B.make_config(base.replace(recompute_mask=0b111111)))
    assert rc0 == 0 and rc3 > 0 and rca == 2 * rc3
    # recomputing 3 of 6 blocks frees the activations of 3 blocks from the per-handle
    # workspace and adds one transient set for the forward pass (the recomputation
    # leaves out FC2, whose output is the checkpointed next-block input)
    act = rc3 // 3
    assert ws0 - ws3 == 3 * act - act
    assert ws3 > 0 and wsa < ws3


def test_create_rejects_bad_arguments_without_gpu():
    lib = B.lib()
    cfg = B.make_config(synth.TINY)
    ws, rc = B.workspace_bytes(cfg)
    h = ctypes.c_void_p()
    assert lib.merak_stage_create(ctypes.byref(cfg), None, ws, None, 0, ctypes.byref(h)) == -1
    assert lib.merak_stage_create(ctypes.byref(cfg), 0x1000 + 16, ws, None, 0, ctypes.byref(h)) == -4
    assert lib.merak_stage_create(ctypes.byref(cfg), 0x100000, ws - 1, None, 0, ctypes.byref(h)) == -5
    cfg_rc = B.make_config(synth.TINY.replace(recompute_mask=1))
    ws, rc = B.workspace_bytes(cfg_rc)
    assert rc > 0
    assert lib.merak_stage_create(ctypes.byref(cfg_rc), 0x100000, ws, None, rc, ctypes.byref(h)) == -1
    assert lib.merak_stage_create(ctypes.byref(cfg_rc), 0x100000, ws, 0x200000, rc - 1, ctypes.byref(h)) == -5
    bad = B.make_config(synth.TINY.replace(seq_len=100))
    assert lib.merak_stage_create(ctypes.byref(bad), 0x100000, ws, None, 0, ctypes.byref(h)) == -2
    assert lib.merak_stage_create(ctypes.byref(cfg), 0x100000, ws, None, 0, None) == -1


def test_stage_calls_reject_null_handle():
    lib = B.lib()
    assert lib.merak_stage_fwd(None, 0x1000, 0x1000, 0x1000, None, None, None) == -1
    assert lib.merak_stage_recompute(None, 0x1000, None, None) == -1
    assert lib.merak_stage_bwd(None, 0x1000, 0x1000, 0x1000, 0x1000, 0, None, None, None) == -1
    assert lib.merak_stage_destroy(None) == -1


def test_kernel_entry_points_validate_before_launch():
    lib = B.lib()
    p = 0x100000
    # M not a multiple of 64
    assert lib.merak_gemm(0, 0, 0, 0, 100, 64, 64, p, 64, p, 64, p, None, None, None, 0, None) == -2
    # bad epilogue / flags / dtype
    assert lib.merak_gemm(0, 0, 0, 9, 64, 64, 64, p, 64, p, 64, p, None, None, None, 0, None) == -1
    assert lib.merak_gemm(0, 2, 0, 0, 64, 64, 64, p, 64, p, 64, p, None, None, None, 0, None) == -1
    assert lib.merak_gemm(3, 0, 0, 0, 64, 64, 64, p, 64, p, 64, p, None, None, None, 0, None) == -1
    # bias epilogue without bias, misaligned operand, lda too small
    assert lib.merak_gemm(0, 0, 0, 1, 64, 64, 64, p, 64, p, 64, p, None, None, None, 0, None) == -1
    assert lib.merak_gemm(0, 0, 0, 0, 64, 64, 64, p + 2, 64, p, 64, p, None, None, None, 0, None) == -4
    assert lib.merak_gemm(0, 0, 0, 0, 64, 64, 128, p, 64, p, 128, p, None, None, None, 0, None) == -2
    assert lib.merak_attention_fwd(0, 1, 100, 1, 64, p, p, p, None) == -2
    assert lib.merak_attention_fwd(0, 1, 128, 1, 80, p, p, p, None) == -7
    assert lib.merak_layernorm_fwd(0, 4, 12, 1e-5, p, p, p, p, p, p, None) == -2
    assert lib.merak_column_sum(0, 4, 64, p, p, 2, p, None) == -1
    assert B.reduce_scratch_elems(128, 10) == 2 * 10
    assert B.reduce_scratch_elems(0, 10) == 0


def test_gemm_rejects_operands_beyond_its_offsets():
    """bf16 operands past 2^31 bytes (with 256 rows of padding) are a shape error, found
    before any launch; the fp32 kernel indexes with 64 bits."""
    lib = B.lib()
    p = 0x100000
    assert lib.merak_gemm(0, 0, 0, 0, 1 << 19, 64, 2048, p, 2048, p, 2048, p, None, None, None, 0, None) == -2
    assert lib.merak_gemm(0, 1, 0, 0, 64, 64, 1 << 20, p, 1024, p, 1 << 20, p, None, None, None, 0, None) == -2


def test_count_nonfinite_validates_before_launch():
    lib = B.lib()
    p = 0x100000
    assert lib.merak_count_nonfinite(2, p, 16, p, None) == -1      # dtype
    assert lib.merak_count_nonfinite(0, p, -1, p, None) == -2      # negative size
    assert lib.merak_count_nonfinite(0, p, 16, None, None) == -1   # no count
    assert lib.merak_count_nonfinite(0, None, 16, p, None) == -1   # no input
    assert lib.merak_count_nonfinite(0, p + 2, 16, p, None) == -4  # misaligned input


def test_kernel_entry_points_reject_empty_inputs():
    """A size of 0 is refused before anything is launched (no GPU needed)."""
    lib = B.lib()
    p = 0x100000
    for M, N, K in ((0, 64, 64), (64, 0, 64), (64, 64, 0)):
        assert lib.merak_gemm(0, 0, 0, 0, M, N, K, p, 64, p, 64, p, None, None, None, 0, None) == -2
    assert lib.merak_layernorm_fwd(0, 0, 64, 1e-5, p, p, p, p, p, p, None) == -2
    assert lib.merak_layernorm_bwd(0, 0, 64, p, p, p, p, p, p, p, p, p, 0, p, None) == -2
    assert lib.merak_layernorm_bwd_noalloc(0, 0, 64, p, p, p, p, p, p, p, p, p, 0, None) == -2
    assert lib.merak_column_sum(0, 0, 64, p, p, 0, p, None) == -2
    for batch, seq, heads in ((0, 64, 1), (1, 0, 1), (1, 64, 0)):
        assert lib.merak_attention_fwd(0, batch, seq, heads, 64, p, p, p, None) == -2
        assert lib.merak_attention_bwd(0, batch, seq, heads, 64, p, p, p, p, p, p, None) == -2
