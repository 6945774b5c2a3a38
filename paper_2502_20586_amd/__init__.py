"""MXFP4 backward-pass hot path of "Training LLMs with MXFP4" for AMD MI355X (gfx950).

Thin Python binding over the C ABI of ``libmxfp4.so`` (see include/mxfp4.h).
Every function marshals torch device tensors into pointers and sizes and calls
the library; all arithmetic runs in the library's HIP kernels. There is no
fallback: if the library is missing or the device is not gfx950 the calls
raise.
"""

from .binding import (MX_BWD_ACCUMULATE, MX_BWD_DX_BF16, MX_MODE_NR, MX_MODE_RHT_NR, MX_MODE_RHT_SR,
                      MX_MODE_SR, MX_MODE_RHT_SR8, MX_NOALLOC_SCRATCH_BYTES, MxError, lib_path, load_library, mx_gemm_f4, mx_gemm_f4_workspace_bytes, mx_release_workspace,
                      mx_linear_backward, mx_linear_backward_noalloc,
                      mx_linear_backward_ex, mx_linear_backward_ex_workspace_bytes, mx_linear_backward_mode,
                      mx_linear_backward_workspace_bytes, mx_measure_mfma_peak, mx_profile_start, mx_profile_stop, mx_quantize,
                      mx_quantize_pair,
                      mx_rht_sr_quantize, mx_rht_sr_quantize_t, quantized_shapes)

__all__ = [
    "MX_MODE_RHT_SR", "MX_MODE_SR", "MX_MODE_RHT_NR", "MX_MODE_NR", "MX_BWD_DX_BF16", "MX_BWD_ACCUMULATE",
    "MX_NOALLOC_SCRATCH_BYTES", "mx_linear_backward_noalloc", "MX_MODE_RHT_SR8",
    "MxError", "lib_path", "load_library",
    "mx_rht_sr_quantize", "mx_rht_sr_quantize_t", "mx_quantize", "mx_quantize_pair", "mx_gemm_f4", "mx_gemm_f4_workspace_bytes", "mx_release_workspace", "mx_linear_backward",
    "mx_linear_backward_mode", "mx_linear_backward_workspace_bytes", "mx_linear_backward_ex",
    "mx_linear_backward_ex_workspace_bytes", "mx_measure_mfma_peak", "mx_profile_start", "mx_profile_stop",
    "quantized_shapes",
]
