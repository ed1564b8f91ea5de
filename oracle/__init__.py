"""CPU oracle for the W4A4 linear (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package.  It never imports the HIP library or its Python binding.
"""

from .w4a4 import (  # noqa: F401
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    row_absmax,
    row_scale,
    quantize_rows,
    pack_int4,
    unpack_int4,
    quantize_act,
    pack_weight_int4,
    code_gemm,
    brute_force_gemm,
    epilogue,
    w4a4_gemm,
    w4a4_gemm_i32,
    w4a4_linear,
    w4a4_linear_rows,
)
from .w158a4 import (  # noqa: F401
    ternary_scale,
    quantize_ternary,
    pack_ternary,
    unpack_ternary,
    pack_weight_ternary,
    w158a4_gemm,
    w158a4_gemm_i32,
    w158a4_linear,
    w158a4_linear_rows,
)
from .w4a4_group import (  # noqa: F401
    GROUP_SIZES,
    quantize_rows_group,
    quantize_act_group,
    pack_weight_int4_group,
    group_code_gemm,
    group_sum,
    group_epilogue,
    w4a4g_gemm_f32,
    w4a4g_gemm,
    w4a4g_linear,
    w4a4g_linear_rows,
)
