"""MI355X (gfx950) block-scaled FP8 attention with Delta-Matching.

The computation lives in libattn_fp8.so (C ABI: include/attn_fp8.h, HIP
kernels in csrc/); `binding` marshals torch tensors into it, `synth` draws
the seeded synthetic workloads.
"""
from .binding import (DELTA_CONSISTENT_DO, DELTA_MATCHING, DELTA_MATCHING_COMPENSATED, DELTA_STALE_ROWSUM,
                      FLAG_PBWD_BLOCK_SCALED, FLAG_PROTECTED_DP, FLAG_ISOLATE3,
                      QUANT_BOTH, QUANT_COL, QUANT_ROW, ROWSTATS, RS_MAX_PDP, RS_MAXABS_DS, RS_SUM_DS,
                      RS_SUM_DSCAST, RS_SUM_PCAST, RS_SUMABS_DS, RS_SUMABS_DSCAST, MX, AttnFp8Error, Problem,
                      attn_fp8_bwd, attn_fp8_bwd_noalloc, attn_fp8_bwd_protected_dp, attn_fp8_bwd_workspace_size, attn_fp8_delta, attn_fp8_fwd,
                      attn_fp8_quantize, attn_fp8_quantize_producer, last_error, lib)

__all__ = ["DELTA_CONSISTENT_DO", "DELTA_MATCHING", "DELTA_MATCHING_COMPENSATED", "DELTA_STALE_ROWSUM",
           "FLAG_PBWD_BLOCK_SCALED", "FLAG_PROTECTED_DP", "FLAG_ISOLATE3",
           "QUANT_BOTH", "QUANT_COL", "QUANT_ROW", "ROWSTATS", "RS_MAX_PDP", "RS_MAXABS_DS", "RS_SUM_DS",
           "RS_SUM_DSCAST", "RS_SUM_PCAST", "RS_SUMABS_DS", "RS_SUMABS_DSCAST", "MX", "AttnFp8Error", "Problem",
           "attn_fp8_bwd", "attn_fp8_bwd_noalloc", "attn_fp8_bwd_protected_dp", "attn_fp8_bwd_workspace_size", "attn_fp8_delta", "attn_fp8_fwd",
           "attn_fp8_quantize", "attn_fp8_quantize_producer", "last_error", "lib"]
