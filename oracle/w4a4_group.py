"""CPU oracle for the group-wise W4A4 linear layer.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the test suite, the smoke check in the package entry
file and the CPU-baseline leg of the benchmark use it.  It shares no code with
the HIP library and imports nothing from the package.

What it computes
----------------
The paper's own W4A4 runs quantise in groups along K: group128 for the DiT
and ELF models and group64 ("block/group64") for FLUX (appendix
experimental-details tables, quantization-function rows; the FLUX setting
paragraph of Sec. 4.2).  The operator stays plain (Sec. 3.1; FAQ Q7).  The
paper prints no formula; this oracle extends the per-token reading of the
W4A4 oracle to groups of G consecutive k (G in {64, 128}):

  1. a[r,g]   = max_{k in group g} |x[r,k]|
  2. s[r,g]   = fl32(a[r,g] / 7)                     (IEEE fp32 division)
  3. q[r,k]   = clamp(rne(fl32(x[r,k] / s[r,g(k)])), -8, 7), q = 0 where s = 0
  4. packing as in the W4A4 oracle (even k in the low nibble)
  5. the same on the rows of W[N,K], with scales s_w[n,g]
  6. acc[m,n,g] = sum_{k in group g} q_x[m,k] * q_w[n,k]      (exact integer)
  7. S[m,n] = 0; for g = 0, 1, ...:  S = fl32(S + fl32(fl32(f32(acc[m,n,g]) * s_x[m,g]) * s_w[n,g]))
  8. y[m,n] = bf16_rne(fl32(S + bias[n]))

Every fp32 operation is rounded on its own (no fused multiply-add), and the
groups are added in increasing k order starting from +0.  With one group
(G = K) steps 7-8 reduce to the per-token epilogue exactly (0 + t = t).
Scales are stored [rows, K/G] row-major.
"""

import numpy as np

from .w4a4 import DENOM, QMAX, QMIN, bf16_bits_to_f32, f32_to_bf16_bits, pack_int4, unpack_int4

GROUP_SIZES = (64, 128)


def quantize_rows_group(x_bits, G):
    """Steps 1-3 on a [R, K] bf16 matrix: returns (codes int8 [R,K], scales float32 [R, K/G])."""
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    R, K = x_bits.shape
    assert K % G == 0
    xf = bf16_bits_to_f32(x_bits).reshape(R, K // G, G)
    a = np.max(np.abs(xf), axis=2).astype(np.float32)
    s = (a / DENOM).astype(np.float32)
    q = np.zeros(xf.shape, dtype=np.int8)
    nz = s != 0
    if np.any(nz):
        with np.errstate(over="ignore", under="ignore"):
            quot = (xf[nz] / s[nz][:, None]).astype(np.float32)
        q[nz] = np.clip(np.rint(quot), QMIN, QMAX).astype(np.int8)
    return q.reshape(R, K), s


def quantize_act_group(x_bits, G):
    """Activation path: bf16 [M,K] -> (packed uint8 [M,K/2], scales fp32 [M,K/G])."""
    q, s = quantize_rows_group(x_bits, G)
    return pack_int4(q), s


def pack_weight_int4_group(w_bits, G):
    """Weight path: bf16 [N,K] -> (packed uint8 [N,K/2], scales fp32 [N,K/G])."""
    q, s = quantize_rows_group(w_bits, G)
    return pack_int4(q), s


def group_code_gemm(qx, qw, G):
    """acc[m,n,g] = sum_{k in group g} qx[m,k] * qw[n,k], exact, as int64 [M,N,K/G].

    Each group is a float64 matrix product of integer codes (every partial sum
    is an integer far below 2^53, so it is exact).
    """
    qx = np.asarray(qx)
    qw = np.asarray(qw)
    K = qx.shape[1]
    assert qw.shape[1] == K and K % G == 0
    out = np.empty((qx.shape[0], qw.shape[0], K // G), dtype=np.int64)
    for g in range(K // G):
        sl = slice(g * G, (g + 1) * G)
        out[:, :, g] = (qx[:, sl].astype(np.float64) @ qw[:, sl].astype(np.float64).T).astype(np.int64)
    return out


def group_sum(acc, s_x, s_w):
    """Step 7: S[m,n] = sequential fp32 sum over groups of fl32(fl32(f32(acc) * s_x) * s_w)."""
    acc = np.asarray(acc)
    s_x = np.asarray(s_x, dtype=np.float32)
    s_w = np.asarray(s_w, dtype=np.float32)
    M, N, ng = acc.shape
    assert s_x.shape == (M, ng) and s_w.shape == (N, ng)
    assert np.all(np.abs(acc) < 2 ** 24)
    S = np.zeros((M, N), dtype=np.float32)
    with np.errstate(over="ignore", under="ignore", invalid="ignore"):
        for g in range(ng):
            t = acc[:, :, g].astype(np.float32)
            t = (t * s_x[:, g][:, None]).astype(np.float32)
            t = (t * s_w[:, g][None, :]).astype(np.float32)
            S = (S + t).astype(np.float32)
    return S


def group_epilogue(S, bias_bits=None):
    """Step 8: y = bf16_rne(fl32(S + bias)); no bias leaves S unchanged."""
    S = np.asarray(S, dtype=np.float32)
    if bias_bits is not None:
        with np.errstate(over="ignore", invalid="ignore"):
            S = (S + bf16_bits_to_f32(bias_bits)[None, :]).astype(np.float32)
    return f32_to_bf16_bits(S)


def w4a4g_gemm_f32(qx_packed, s_x, qw_packed, s_w, G):
    """Steps 6-7 on packed operands: the fp32 group sum S [M,N] before bias and bf16 rounding."""
    acc = group_code_gemm(unpack_int4(qx_packed), unpack_int4(qw_packed), G)
    return group_sum(acc, s_x, s_w)


def w4a4g_gemm(qx_packed, s_x, qw_packed, s_w, G, bias_bits=None):
    """Steps 6-8 on packed operands: bf16 bits [M,N]."""
    return group_epilogue(w4a4g_gemm_f32(qx_packed, s_x, qw_packed, s_w, G), bias_bits)


def w4a4g_linear(x_bits, qw_packed, s_w, G, bias_bits=None):
    """Full group-wise layer on bf16 activations and a pre-packed weight: bf16 bits [M,N]."""
    qx, s_x = quantize_act_group(x_bits, G)
    return w4a4g_gemm(qx, s_x, qw_packed, s_w, G, bias_bits)


def w4a4g_linear_rows(x_bits, qw_packed, s_w, G, rows, bias_bits=None):
    """The layer's output for a subset of rows only (quantisation is row-local)."""
    rows = np.asarray(rows)
    return w4a4g_linear(np.asarray(x_bits)[rows], qw_packed, s_w, G, bias_bits)
