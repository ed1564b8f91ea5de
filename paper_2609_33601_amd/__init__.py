"""MI355X (gfx950) W4A4 linear: per-token int4 activation quantisation, packed
int4 x int4 GEMM on int8 MFMA with exact int32 accumulation, fused dequantising
epilogue.  The kernels live in libjq.so (C ABI in include/jq.h); this package is
its Python binding plus the seeded workload generators.
"""

from .jq import (  # noqa: F401
    JQError,
    bf16_bits,
    bf16_tensor,
    jq_pack_weight_int4,
    jq_quantize_act,
    jq_status_string,
    jq_version,
    jq_w4a4_gemm,
    jq_w4a4_gemm_i32,
    jq_w4a4_linear,
    jq_w4a4_workspace_bytes,
    lib,
)
