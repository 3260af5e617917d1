"""Kernel classes of the stage step: the library's timing classes
(merak_stage_set_timing), what each launch covers, and which kernel names in a
rocprofv3 trace or counter file belong to each class.

A GEMM instantiation's template tail names its layout and epilogue:
``gemm_mfma_kernel<BM, BN, WM, WN, NS, A_T, B_T, EPI>``.  Forward GEMMs read
both operands along K (A_T = B_T = false), input-gradient GEMMs read the weight
in place (B_T = true), weight-gradient GEMMs read both operands transposed and
write fp32 (A_T = B_T = true, EPI 5).  The two weight-gradient launches of a
block share an instantiation; the FC1/FC2 launch has the larger grid."""
from __future__ import annotations

from . import binding as B

CLASSES = {
    # name: (timing class id, description of one launch)
    "GEMM_FWD": (B.KC_GEMM_FWD, "forward GEMMs (QKV, projection, FC1, FC2; recompute too), one grouped launch "
                                "per step and stream"),
    "GEMM_DX": (B.KC_GEMM_DX, "input-gradient GEMMs (FC2 with GeLU', FC1, projection, QKV), one grouped launch "
                              "per step and stream"),
    "GEMM_DW": (B.KC_GEMM_DW, "weight-gradient GEMM of FC1 and FC2 of one block (grouped, fp32 out)"),
    "GEMM_DW_ATTN": (B.KC_GEMM_DW_ATTN, "weight-gradient GEMM of QKV and the projection of one block "
                                        "(grouped, fp32 out)"),
    "ATTN_FWD": (B.KC_ATTN_FWD, "causal attention forward, one grouped launch per stream"),
    "ATTN_BWD": (B.KC_ATTN_BWD, "attention backward (dQ with delta, then dK/dV), one grouped pair per stream"),
    "LN_FWD": (B.KC_LN_FWD, "LayerNorm forward"),
    "LN_BWD": (B.KC_LN_BWD, "LayerNorm backward with the residual gradient"),
    "REDUCE": (B.KC_REDUCE, "bias and LayerNorm-parameter gradient sums (partials, then their sum)"),
}


def classify(kernel_name: str, grid: int, dw_grids: tuple = ()) -> str | None:
    """Class of one dispatch in a rocprofv3 trace; `dw_grids` lists the grid
    sizes of the weight-gradient GEMM dispatches seen, the largest being FC1/FC2."""
    n = kernel_name
    if "gemm_mfma_kernel" in n or "gemm_f32_kernel" in n:
        tail = n[n.index("<"):] if "<" in n else ""
        parts = [p.strip(" <>()") for p in tail.split(",")]
        a_t, b_t = parts[-3] == "true", parts[-2] == "true"
        if a_t and b_t:
            return "GEMM_DW" if (not dw_grids or grid == max(dw_grids)) else "GEMM_DW_ATTN"
        return "GEMM_DX" if b_t else "GEMM_FWD"
    if "attn_fwd" in n:
        return "ATTN_FWD"
    if "attn_bwd" in n or "attn_delta" in n:
        return "ATTN_BWD"
    if "ln_fwd_kernel" in n:
        return "LN_FWD"
    if "ln_bwd_kernel" in n:
        return "LN_BWD"
    if "partials_kernel" in n:
        return "REDUCE"
    return None


def is_dw(kernel_name: str) -> bool:
    return "gemm_mfma_kernel" in kernel_name and "true, true, 5>" in kernel_name
