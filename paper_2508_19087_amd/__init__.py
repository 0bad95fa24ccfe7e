"""WpAq bipolar-INT bit-plane integer GEMM for AMD MI355X (gfx950).

An MI355X-native implementation of the arbitrary-precision integer matrix
multiply of APT-LLM (arXiv 2508.19087): signed-INT codes are converted to
bipolar-INT, split into bit-planes packed in HBM, and multiplied exactly into
an int32 result with an optional fp16 scale epilogue.  The computation lives in
hand-written HIP kernels behind the C ABI of include/apt.h (libapt.so); this
package is its Python binding.
"""
from .apt import (APT_ACT_CODES, APT_ACT_FP16, APT_DECODE_MAX_M, APT_ERR_HIP, APT_ERR_INVALID_ARG, APT_ERR_UNSUPPORTED, APT_ERR_WORKSPACE,  # noqa: F401
                  APT_OK, APT_ROUTE_AUTO, APT_ROUTE_FP4_MFMA, APT_ROUTE_FP6_MFMA, APT_ROUTE_FP8_MFMA, APT_ROUTE_INT8_MFMA, APT_ROUTE_PM1_MFMA, APT_ROUTE_XOR,
                  ROUTE_NAMES, AptError, Packed, apt_config_t, apt_gemm, apt_gemm_affine,
                  apt_gemm_workspace_bytes, apt_config_table_clear, apt_config_table_size,
                  apt_last_hip_error, apt_gemm_noalloc, apt_gemm_decode, gemm_decode,
                  apt_gemm_act, apt_gemm_act_workspace_bytes, gemm_act,
                  apt_search_config, apt_search_workspace_bytes, check,
                  apt_pack_weights, apt_packed_bytes, apt_quantize_pack_activations,
                  apt_quantize_pack_activations_fp16, apt_select_config, gemm, header_functions,
                  gemm_affine, lib, pack, quantize_pack, search_config, select_config,
                  status_string)
