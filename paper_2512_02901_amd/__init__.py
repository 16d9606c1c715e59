"""Fairy2i quantised widely-linear layer on MI355X (gfx950).

The computation lives in libfairy2i.so (HIP kernels behind the C ABI of
include/fairy2i.h); this package only marshals torch device tensors into it.
Importing the package does not load the library; the first call does, and
raises if it has not been built (there is no fallback path).
"""
from .binding import (ACT_BF16, ACT_F32, ACT_I8, LAYOUT_D3, LAYOUT_TILED, LAYOUT_TILED_FP4,  # noqa: F401
                      MAX_DECODE_BATCH, MAX_STAGES, PROBE_MFMA_F8F4, PROBE_MFMA_I8, PROBE_MFMA_I8_32X32, Fairy2iError, WlBlock, WlGroup, cpu_lut_wl_matmul,
                      cpu_lut_workspace_bytes, cgemm_gauss, cgemm_gauss_planar_workspace_bytes, int8_accumulators, load, qat_fake_quant,
                      probe_mfma, qat_ste_backward, quantize, quantize_grouped,
                      quantize_act_int8, repack_tiled, repack_tiled_bytes, repack_tiled_fp4, to_widely_linear,
                      wl_matmul, wl_matmul_noalloc, wl_matmul_workspace_bytes, wl_realify, wl_realify_codes, wl_unrealify_grad,
                      f32_to_bf16, gemm_bf16)

__all__ = [
    "to_widely_linear", "quantize", "quantize_grouped", "quantize_act_int8", "wl_matmul", "wl_matmul_noalloc", "int8_accumulators",
    "wl_matmul_workspace_bytes", "repack_tiled", "repack_tiled_fp4", "repack_tiled_bytes", "load",
    "Fairy2iError", "WlBlock", "WlGroup", "ACT_F32", "ACT_BF16", "ACT_I8", "LAYOUT_D3", "LAYOUT_TILED",
    "LAYOUT_TILED_FP4", "MAX_STAGES", "MAX_DECODE_BATCH", "cpu_lut_wl_matmul", "cpu_lut_workspace_bytes",
    "qat_fake_quant", "qat_ste_backward", "cgemm_gauss", "cgemm_gauss_planar_workspace_bytes",
    "probe_mfma", "PROBE_MFMA_I8", "PROBE_MFMA_F8F4", "PROBE_MFMA_I8_32X32", "wl_realify", "wl_realify_codes", "wl_unrealify_grad",
    "f32_to_bf16", "gemm_bf16",
]
