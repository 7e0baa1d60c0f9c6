"""MI355X (gfx950) implementation of FQ-ViT's integer hot path: PTF LayerNorm
and Log-Int-Softmax attention with BitShift Attn x V.

The computation lives in libfqvit.so (HIP kernels behind the C ABI of
include/fqvit.h); this package only builds and binds it.
"""
from .binding import (FqError, codes_ld, lis_attention_head, lis_attention_qk,  # noqa: F401
                      lis_attn_v_shift, lis_attn_v_shift_wide,
                      lis_softmax_log4, ptf_calibrate, ptf_calibrate_noalloc,
                      ptf_calibrate_workspace_bytes,
                      ptf_layernorm_int8, ptf_quantize_int8, requant_dyadic_int8, status_str,
                      time_next_call,
                      version)

__all__ = ["ptf_layernorm_int8", "lis_softmax_log4", "lis_attn_v_shift", "lis_attn_v_shift_wide",
           "lis_attention_head",
           "lis_attention_qk",
           "ptf_calibrate", "ptf_calibrate_noalloc", "ptf_calibrate_workspace_bytes",
           "ptf_quantize_int8",
           "requant_dyadic_int8", "FqError", "codes_ld", "status_str", "time_next_call",
           "version"]
