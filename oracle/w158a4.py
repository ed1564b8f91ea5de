"""CPU oracle for the W1.58A4 linear layer: ternary weights, int4 activations.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the test suite, the smoke check in the package entry
file and the CPU-baseline leg of the benchmark use it.  It shares no code with
the HIP library and imports nothing from the package.

What it computes
----------------
Ternary (1.58-bit) weights with INT4 activations is the paper's most-featured
deployment setting: the W1.58A4 rows of the DiT and ELF result tables (Sec. 4)
and the "Ternary weights, INT4 activations" quantization-function rows of the
appendix experimental-details tables.  As for W4A4, the deployed operator is
plain (Sec. 3.1; appendix FAQ Q7): quantise, pack, low-bit matrix multiply,
dequantise.  The activation side is the per-token int4 path of the W4A4
oracle, unchanged.  The paper prints no formula for the ternary weight
quantiser; this oracle fixes the absmean reading used by the ternary-weight
systems the paper builds on (the ternary DiT and language-model baselines it
compares against), one scale per output channel:

  1. S[n] = sum_k |w[n,k]|                    (float64)
     g[n] = fl32(fl64(S[n] / K))              (fp64 IEEE division, then RNE to fp32)
  2. t[n,k] = clamp(rne(fl32(w[n,k] / g[n])), -1, 1), and t = 0 when g = 0
  3. pack: byte j of row n holds codes 4j .. 4j+3; code 4j+i sits in bits
     2i .. 2i+1 as a two's-complement 2-bit field (0 -> 00, 1 -> 01, -1 -> 11)
  4. acc[m,n] = sum_k q_x[m,k] * t[n,k]       (exact integer)
  5. y[m,n] = bf16_rne(((fl32(acc) * s_x[m]) * g[n]) + bias[n]), the W4A4
     epilogue with g as the per-channel weight scale.

The float64 sum in step 1 is exact (hence independent of summation order)
whenever a row's nonzero magnitudes span less than 2^29: each bf16 value
carries 8 significant bits and K <= 2^16 adds at most 16 more, which fits the
53-bit float64 significand.  Real weight rows are far inside that range.
"""

import numpy as np

from .w4a4 import bf16_bits_to_f32, code_gemm, epilogue, quantize_act, unpack_int4

TMIN, TMAX = -1, 1


def ternary_scale(w_bits):
    """Step 1: g[n] = fl32(fl64(sum_k |w[n,k]|) / K), one scale per row."""
    w_bits = np.asarray(w_bits, dtype=np.uint16)
    assert w_bits.ndim == 2
    K = w_bits.shape[1]
    wf = bf16_bits_to_f32(w_bits).astype(np.float64)
    S = np.sum(np.abs(wf), axis=1, dtype=np.float64)
    return (S / np.float64(K)).astype(np.float32)


def quantize_ternary(w_bits):
    """Steps 1-2 on a [N, K] bf16 weight: returns (codes int8 [N,K] in {-1,0,1}, scale float32 [N])."""
    w_bits = np.asarray(w_bits, dtype=np.uint16)
    wf = bf16_bits_to_f32(w_bits)
    g = ternary_scale(w_bits)
    t = np.zeros(wf.shape, dtype=np.int8)
    nz = g != 0
    if np.any(nz):
        with np.errstate(over="ignore", under="ignore"):
            quot = (wf[nz] / g[nz, None]).astype(np.float32)
        t[nz] = np.clip(np.rint(quot), TMIN, TMAX).astype(np.int8)
    return t, g


def pack_ternary(t):
    """Step 3: codes [N, K] (K % 4 == 0) -> bytes [N, K/4], code 4j+i in bits 2i..2i+1."""
    t = np.asarray(t, dtype=np.int16)
    assert t.ndim == 2 and t.shape[1] % 4 == 0
    out = np.zeros((t.shape[0], t.shape[1] // 4), dtype=np.int16)
    for i in range(4):
        out |= (t[:, i::4] & 0x3) << (2 * i)
    return out.astype(np.uint8)


def unpack_ternary(packed):
    """Inverse of pack_ternary: bytes [N, K/4] -> int8 codes [N, K] (two's-complement 2-bit fields)."""
    p = np.asarray(packed, dtype=np.uint8).astype(np.int16)
    out = np.empty((p.shape[0], p.shape[1] * 4), dtype=np.int8)
    for i in range(4):
        f = (p >> (2 * i)) & 0x3
        out[:, i::4] = np.where(f >= 2, f - 4, f)
    return out


def pack_weight_ternary(w_bits):
    """Weight path: bf16 W [N,K] -> (packed uint8 [N,K/4], scale fp32 [N])."""
    t, g = quantize_ternary(w_bits)
    return pack_ternary(t), g


def w158a4_gemm(qx_packed, s_x, wt_packed, g, bias_bits=None):
    """Steps 4-5 on packed operands (int4 activations, ternary weights): bf16 bits [M,N]."""
    acc = code_gemm(unpack_int4(qx_packed), unpack_ternary(wt_packed))
    return epilogue(acc, s_x, g, bias_bits)


def w158a4_gemm_i32(qx_packed, wt_packed):
    """Step 4 only: exact accumulators as int32 [M,N]."""
    return code_gemm(unpack_int4(qx_packed), unpack_ternary(wt_packed)).astype(np.int32)


def w158a4_linear(x_bits, wt_packed, g, bias_bits=None):
    """Full layer on bf16 activations and a pre-packed ternary weight: bf16 bits [M,N]."""
    qx, s_x = quantize_act(x_bits)
    return w158a4_gemm(qx, s_x, wt_packed, g, bias_bits)


def w158a4_linear_rows(x_bits, wt_packed, g, rows, bias_bits=None):
    """The layer's output for a subset of rows only (activation quantisation is row-local)."""
    rows = np.asarray(rows)
    return w158a4_linear(np.asarray(x_bits)[rows], wt_packed, g, bias_bits)
