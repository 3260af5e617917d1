"""ctypes binding of libmerak_stage.so (argument marshalling only).

Every step of the forward, recompute and backward passes runs in the HIP
library; this module only converts Python arguments to the C ABI of
``include/merak_stage.h``.  PyTorch supplies device memory and streams.
If the library is missing the calls raise: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import synth

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmerak_stage.so")
PARAMS_PER_BLOCK = 12
BF16, FP32 = 0, 1

STATUS = {0: "MERAK_OK", -1: "MERAK_ERR_INVALID_ARG", -2: "MERAK_ERR_SHAPE", -3: "MERAK_ERR_ORDER",
          -4: "MERAK_ERR_ALIGN", -5: "MERAK_ERR_WORKSPACE", -6: "MERAK_ERR_HIP", -7: "MERAK_ERR_UNSUPPORTED"}

EPI_STORE, EPI_BIAS, EPI_BIAS_GELU, EPI_BIAS_RESID, EPI_GELU_BWD, EPI_F32 = range(6)
(KC_NONE, KC_GEMM_FWD, KC_GEMM_DX, KC_GEMM_DW, KC_ATTN_FWD, KC_ATTN_BWD, KC_LN_FWD, KC_LN_BWD,
 KC_REDUCE, KC_GEMM_DW_ATTN) = range(10)


class MerakError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {STATUS.get(status, status)}")
        self.status = status


class StageConfig(ctypes.Structure):
    _fields_ = [("n_blocks", ctypes.c_int32), ("hidden", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("ffn", ctypes.c_int32), ("seq_len", ctypes.c_int32), ("micro_batch", ctypes.c_int32),
                ("tp_degree", ctypes.c_int32), ("n_sub_microbatches", ctypes.c_int32),
                ("recompute_mask", ctypes.c_uint64), ("dtype", ctypes.c_int32), ("ln_eps", ctypes.c_float)]


_lib = None
_P, _I, _SZ, _F = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_float
_SIGS = {
    "merak_status_str": ([_I], ctypes.c_char_p),
    "merak_stage_validate": ([ctypes.POINTER(StageConfig)], _I),
    "merak_stage_param_layout": ([ctypes.POINTER(StageConfig), ctypes.POINTER(_SZ), _P], _I),
    "merak_stage_workspace_bytes": ([ctypes.POINTER(StageConfig), ctypes.POINTER(_SZ), ctypes.POINTER(_SZ)], _I),
    "merak_stage_create": ([ctypes.POINTER(StageConfig), _P, _SZ, _P, _SZ, ctypes.POINTER(_P)], _I),
    "merak_stage_destroy": ([_P], _I),
    "merak_stage_fwd": ([_P, _P, _P, _P, _P, _P, _P], _I),
    "merak_stage_recompute": ([_P, _P, _P, _P], _I),
    "merak_stage_bwd": ([_P, _P, _P, _P, _P, _I, _P, _P, _P], _I),
    "merak_stage_set_timing": ([_P, _I], _I),
    "merak_stage_read_timing": ([_P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)], _I),
    "merak_gemm": ([_I, _I, _I, _I, _I, _I, _I, _P, _I, _P, _I, _P, _P, _P, _P, _I, _P], _I),
    "merak_gemm_tile_override": ([_I], _I),
    "merak_plan_recompute": ([_I, ctypes.c_double, _I, _P, _P], _I),
    "merak_schedule_stage": ([_I, _I, _I, _I, _P, _I, ctypes.POINTER(_I)], _I),
    "merak_schedule_simulate": ([_I, _I, _I, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                 ctypes.POINTER(ctypes.c_double), _P], _I),
    "merak_debug_fail_after": ([_I], _I),
    "merak_schedule_inflight": ([_I, _I, _I, _I, ctypes.POINTER(_I)], _I),
    "merak_schedule_run": ([_I, _I, _I, _I, _P, _I, _P, _P, _P, _P, _P, _P, _I, _P, _P], _I),
    "merak_graph_shard": ([_I, _P, _P, _P, _P, _P, _I, _P, _I, _P, ctypes.POINTER(ctypes.c_int32), _P, _P, _I], _I),
    "merak_plan_alpha1": ([_I, ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                           ctypes.POINTER(ctypes.c_double)], _I),
    "merak_layernorm_fwd": ([_I, _I, _I, _F, _P, _P, _P, _P, _P, _P, _P], _I),
    "merak_reduce_scratch_elems": ([_I, _I], _SZ),
    "merak_layernorm_bwd": ([_I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _P, _P], _I),
    "merak_layernorm_bwd_noalloc": ([_I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _P], _I),
    "merak_noalloc_scratch_elems": ([], _SZ),
    "merak_column_sum": ([_I, _I, _I, _P, _P, _I, _P, _P], _I),
    "merak_count_nonfinite": ([_I, _P, ctypes.c_int64, _P, _P], _I),
    "merak_attention_fwd": ([_I, _I, _I, _I, _I, _P, _P, _P, _P], _I),
    "merak_attention_bwd": ([_I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P], _I),
}


def lib() -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2206_04959_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def _check(status: int, what: str) -> None:
    if status != 0:
        raise MerakError(status, what)


def make_config(shape: synth.StageShape) -> StageConfig:
    return StageConfig(shape.n_blocks, shape.hidden, shape.n_heads, shape.ffn, shape.seq_len, shape.micro_batch,
                       shape.tp_degree, shape.n_sub, shape.recompute_mask,
                       BF16 if shape.dtype == "bf16" else FP32, shape.ln_eps)


def validate(cfg: StageConfig) -> int:
    return lib().merak_stage_validate(ctypes.byref(cfg))


def param_layout(cfg: StageConfig):
    """(total elements, offsets [n_blocks, 12])."""
    total = ctypes.c_size_t()
    offs = np.zeros(cfg.n_blocks * PARAMS_PER_BLOCK, dtype=np.uint64)
    _check(lib().merak_stage_param_layout(ctypes.byref(cfg), ctypes.byref(total),
                                          offs.ctypes.data_as(ctypes.c_void_p)), "param_layout")
    return int(total.value), offs.reshape(cfg.n_blocks, PARAMS_PER_BLOCK).astype(np.int64)


def workspace_bytes(cfg: StageConfig):
    ws, rc = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().merak_stage_workspace_bytes(ctypes.byref(cfg), ctypes.byref(ws), ctypes.byref(rc)),
           "workspace_bytes")
    return int(ws.value), int(rc.value)


def pack_params(cfg: StageConfig, blocks: Sequence[Dict[str, np.ndarray]]) -> np.ndarray:
    """Flat host parameter buffer (uint16 bf16 bits or float32) in the library's
    layout from per-block dicts of device-format arrays."""
    total, offs = param_layout(cfg)
    dt = np.uint16 if cfg.dtype == BF16 else np.float32
    flat = np.zeros(total, dtype=dt)
    for l, blk in enumerate(blocks):
        for i, name in enumerate(synth.PARAM_NAMES):
            a = np.ascontiguousarray(blk[name]).ravel()
            flat[offs[l, i]: offs[l, i] + a.size] = a.astype(dt, copy=False)
    return flat


def unpack(cfg: StageConfig, flat: np.ndarray, shape: synth.StageShape) -> List[Dict[str, np.ndarray]]:
    """Per-block dicts of views into a flat buffer laid out like the parameters."""
    _, offs = param_layout(cfg)
    shapes = shape.local_param_shapes()
    out = []
    for l in range(cfg.n_blocks):
        d = {}
        for i, name in enumerate(synth.PARAM_NAMES):
            n = int(np.prod(shapes[name]))
            d[name] = flat[offs[l, i]: offs[l, i] + n].reshape(shapes[name])
        out.append(d)
    return out


# ---------------------------------------------------------------------------
# torch plumbing (device memory and streams)
# ---------------------------------------------------------------------------

def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(s) -> Optional[int]:
    import torch
    if s is None:
        return torch.cuda.current_stream().cuda_stream
    return s.cuda_stream


def to_device(payload: np.ndarray, device="cuda"):
    """Upload a device-format host array (uint16 bf16 bits or float32)."""
    import torch
    if payload.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(payload).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(payload, dtype=np.float32)).to(device)


def to_host_f64(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


class Stage:
    """A handle of the HIP library plus its caller-owned device memory."""

    def __init__(self, shape: synth.StageShape, recompute_area=None, device="cuda"):
        import torch
        self.shape = shape
        self.cfg = make_config(shape)
        ws, rc = workspace_bytes(self.cfg)
        self.workspace_bytes, self.recompute_bytes = ws, rc
        self.workspace = torch.empty(max(ws, 256), dtype=torch.uint8, device=device)
        if rc > 0 and recompute_area is None:
            recompute_area = torch.empty(rc, dtype=torch.uint8, device=device)
        self.recompute_area = recompute_area
        h = ctypes.c_void_p()
        _check(lib().merak_stage_create(ctypes.byref(self.cfg), self.workspace.data_ptr(), ws,
                                        _ptr(recompute_area), rc, ctypes.byref(h)), "merak_stage_create")
        self.handle = h

    def fwd(self, params, x, y, fwd_partials=None, streams=(None, None)) -> None:
        _check(lib().merak_stage_fwd(self.handle, _ptr(params), _ptr(x), _ptr(y), _ptr(fwd_partials),
                                     _stream(streams[0]), _stream(streams[1])), "merak_stage_fwd")

    def recompute(self, params, streams=(None, None)) -> None:
        _check(lib().merak_stage_recompute(self.handle, _ptr(params), _stream(streams[0]), _stream(streams[1])),
               "merak_stage_recompute")

    def bwd(self, params, dy, dx, grads, accumulate=False, bwd_partials=None, streams=(None, None)) -> None:
        _check(lib().merak_stage_bwd(self.handle, _ptr(params), _ptr(dy), _ptr(dx), _ptr(grads), int(accumulate),
                                     _ptr(bwd_partials), _stream(streams[0]), _stream(streams[1])),
               "merak_stage_bwd")

    def set_timing(self, kernel_class: int) -> None:
        _check(lib().merak_stage_set_timing(self.handle, kernel_class), "merak_stage_set_timing")

    def read_timing(self):
        """(total ms, launches) of the timed kernel class since the last read."""
        ms, n = ctypes.c_double(), ctypes.c_int64()
        _check(lib().merak_stage_read_timing(self.handle, ctypes.byref(ms), ctypes.byref(n)),
               "merak_stage_read_timing")
        return float(ms.value), int(n.value)

    def close(self) -> None:
        if getattr(self, "handle", None):
            lib().merak_stage_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------------------
# Per-kernel entry points
# ---------------------------------------------------------------------------

def _dt(t) -> int:
    import torch
    return BF16 if t.dtype == torch.bfloat16 else FP32


def gemm(a, b, c, M, N, K, a_trans=False, b_trans=False, epilogue=EPI_STORE, bias=None, resid=None, aux=None,
         accumulate=False, lda=None, ldb=None, dtype=None, stream=None) -> None:
    dt = _dt(a) if dtype is None else dtype
    lda = lda if lda is not None else (M if a_trans else K)
    ldb = ldb if ldb is not None else (N if b_trans else K)
    _check(lib().merak_gemm(dt, int(a_trans), int(b_trans), epilogue, M, N, K, _ptr(a), lda, _ptr(b), ldb,
                            _ptr(c), _ptr(bias), _ptr(resid), _ptr(aux), int(accumulate), _stream(stream)),
           "merak_gemm")


SCHED_1F1B, SCHED_EARLY_RECOMPUTE, SCHED_SCP = range(3)
OP_FWD, OP_RECOMPUTE, OP_BWD, OP_RECOMPUTE_BWD = range(4)


def schedule_stage(kind: int, n_stages: int, n_micro: int, stage: int):
    """Op list of one stage: [(op type, micro-batch)]."""
    n = ctypes.c_int()
    buf = (ctypes.c_int32 * (3 * n_micro + 4))()
    _check(lib().merak_schedule_stage(kind, n_stages, n_micro, stage, buf, len(buf), ctypes.byref(n)),
           "merak_schedule_stage")
    return [(int(v) >> 24, int(v) & 0xFFFFFF) for v in buf[:n.value]]


def schedule_simulate(kind: int, n_stages: int, n_micro: int, cost_fwd=1.0, cost_rc=1.0, cost_bwd=2.0):
    """(makespan, [busy time per stage]) of the greedy in-order execution."""
    mk = ctypes.c_double()
    busy = (ctypes.c_double * n_stages)()
    _check(lib().merak_schedule_simulate(kind, n_stages, n_micro, cost_fwd, cost_rc, cost_bwd, ctypes.byref(mk), busy),
           "merak_schedule_simulate")
    return float(mk.value), list(busy)


def schedule_inflight(kind: int, n_stages: int, n_micro: int, stage: int) -> int:
    """Handles merak_schedule_run needs for this stage (micro-batches in flight)."""
    n = ctypes.c_int()
    _check(lib().merak_schedule_inflight(kind, n_stages, n_micro, stage, ctypes.byref(n)), "merak_schedule_inflight")
    return int(n.value)


def schedule_run(kind: int, n_stages: int, n_micro: int, stage: int, stages, params, xs, ys, dys, dxs, grads,
                 accumulate=False, streams=(None, None)) -> None:
    """Run one stage's op list through its handles (`stages`: Stage objects)."""
    hs = (ctypes.c_void_p * len(stages))(*[s.handle.value for s in stages])
    arr = lambda ts: (ctypes.c_void_p * len(ts))(*[t.data_ptr() for t in ts])  # noqa: E731
    _check(lib().merak_schedule_run(kind, n_stages, n_micro, stage, hs, len(stages), _ptr(params), arr(xs), arr(ys),
                                    arr(dys), arr(dxs), _ptr(grads), int(accumulate), _stream(streams[0]),
                                    _stream(streams[1])), "merak_schedule_run")


def plan_recompute(n_stages: int, alpha1: float, blocks_per_stage: int):
    """Stage-aware recomputation plan: ([alpha_i], [recompute mask of stage i])."""
    a = (ctypes.c_double * n_stages)()
    m = (ctypes.c_uint64 * n_stages)()
    _check(lib().merak_plan_recompute(n_stages, alpha1, blocks_per_stage, a, m), "merak_plan_recompute")
    return list(a), list(m)


def plan_alpha1(n_stages: int, mem_runtime: float, mem_activation: float, capacity: float, step: float) -> float:
    """Largest feasible alpha_1 on the grid of `step` under the stage memory model."""
    out = ctypes.c_double()
    _check(lib().merak_plan_alpha1(n_stages, mem_runtime, mem_activation, capacity, step, ctypes.byref(out)),
           "merak_plan_alpha1")
    return float(out.value)


def debug_fail_after(launches: int) -> int:
    """Inject a launch failure after `launches` more stage launches (-1: off)."""
    return int(lib().merak_debug_fail_after(int(launches)))


def gemm_tile_override(cfg: int) -> int:
    """Force a bf16 GEMM tile shape (1..10) or restore the built-in choice (0);
    returns the previous setting."""
    prev = int(lib().merak_gemm_tile_override(int(cfg)))
    if prev < 0:
        raise ValueError(f"tile configuration {cfg} out of range")
    return prev


def layernorm_fwd(x, gamma, beta, y, mean, rstd, eps=1e-5, stream=None) -> None:
    rows, h = x.shape[0], x.shape[-1]
    _check(lib().merak_layernorm_fwd(_dt(x), rows, h, eps, _ptr(x), _ptr(gamma), _ptr(beta), _ptr(y), _ptr(mean),
                                     _ptr(rstd), _stream(stream)), "merak_layernorm_fwd")


def reduce_scratch_elems(rows: int, cols: int) -> int:
    return int(lib().merak_reduce_scratch_elems(rows, cols))


def layernorm_bwd(dout, x, mean, rstd, gamma, dres, dx, dgamma, dbeta, scratch, accumulate=False,
                  stream=None) -> None:
    rows, h = x.shape[0], x.shape[-1]
    _check(lib().merak_layernorm_bwd(_dt(x), rows, h, _ptr(dout), _ptr(x), _ptr(mean), _ptr(rstd), _ptr(gamma),
                                     _ptr(dres), _ptr(dx), _ptr(dgamma), _ptr(dbeta), int(accumulate),
                                     _ptr(scratch), _stream(stream)), "merak_layernorm_bwd")


def layernorm_bwd_noalloc(dout, x, mean, rstd, gamma, dres, dx, dgamma, dbeta, accumulate=False,
                          stream=None) -> None:
    rows, h = x.shape[0], x.shape[-1]
    _check(lib().merak_layernorm_bwd_noalloc(_dt(x), rows, h, _ptr(dout), _ptr(x), _ptr(mean), _ptr(rstd),
                                             _ptr(gamma), _ptr(dres), _ptr(dx), _ptr(dgamma), _ptr(dbeta),
                                             int(accumulate), _stream(stream)), "merak_layernorm_bwd_noalloc")


def noalloc_scratch_elems() -> int:
    return int(lib().merak_noalloc_scratch_elems())


def column_sum(x, out, scratch, accumulate=False, stream=None) -> None:
    rows, cols = x.shape
    _check(lib().merak_column_sum(_dt(x), rows, cols, _ptr(x), _ptr(out), int(accumulate), _ptr(scratch),
                                  _stream(stream)), "merak_column_sum")


def count_nonfinite(x, count, stream=None) -> None:
    """Enqueue the count of NaN/Inf elements of tensor x into count (a device int64 tensor of one element)."""
    import torch
    if x.dtype not in (torch.bfloat16, torch.float32) or count.dtype != torch.int64 or count.numel() != 1:
        raise ValueError("count_nonfinite: x bf16 or fp32, count one int64 element")
    _check(lib().merak_count_nonfinite(_dt(x), _ptr(x), x.numel(), _ptr(count), _stream(stream)),
           "merak_count_nonfinite")


def attention_fwd(qkv, o, lse, batch, seq, heads, head_dim, stream=None) -> None:
    _check(lib().merak_attention_fwd(_dt(qkv), batch, seq, heads, head_dim, _ptr(qkv), _ptr(o), _ptr(lse),
                                     _stream(stream)), "merak_attention_fwd")


def attention_bwd(qkv, o, lse, dout, dqkv, delta, batch, seq, heads, head_dim, stream=None) -> None:
    _check(lib().merak_attention_bwd(_dt(qkv), batch, seq, heads, head_dim, _ptr(qkv), _ptr(o), _ptr(lse),
                                     _ptr(dout), _ptr(dqkv), _ptr(delta), _stream(stream)), "merak_attention_bwd")
