"""CPU oracle for the plain W4A4 linear layer.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the test suite, the smoke check in the package entry
file and the CPU-baseline leg of the benchmark use it.  It shares no code with
the HIP library (no kernels, headers, helpers or tables) and imports nothing
from the package.

What it computes
----------------
The paper trains models whose deployed operator stays "plain": every
transformer-block linear becomes a low-bit linear of the target deployment
family, with no smoothing, rotation, normalisation or SVD branch added for the
sake of quantisation (Sec. 3.1 "Quantization as distillation"; appendix FAQ
Q7).  For the W4A4 setting the quantisation function is INT4 weights and
activations (appendix "Experimental Details", quantization-function rows; the
"Naive INT4" rows of the FLUX table in Sec. 4.2 are this operator with no
extra branch).  Executing it needs a quantiser, a nibble packer and a low-bit
matrix multiply (FAQ Q7).  The paper prints no formula for the quantiser, so
this oracle fixes one reading and writes it out as a plain definition:

  1. a[m]   = max_k |x[m,k]|                       (exact in fp32)
  2. s[m]   = fl32(a[m] / 7)                        (IEEE fp32 division, RNE)
  3. q[m,k] = clamp(rne(fl32(x[m,k] / s[m])), -8, 7), and q = 0 when s = 0
  4. pack:  byte j of row m = (q[m,2j] & 0xF) | ((q[m,2j+1] & 0xF) << 4)
  5. the same steps on the rows of W[N,K] (one scale per output channel)
  6. acc[m,n] = sum_k q_x[m,k] * q_w[n,k]           (exact integer)
  7. y[m,n] = bf16_rne(((fl32(acc) * s_x[m]) * s_w[n]) + bias[n])
     in fp32, each operation rounded on its own (no fused multiply-add).

Readings (where the paper is silent): symmetric codes with zero-point 0,
denominator 7 = 2^(4-1) - 1, fp32 scales, true division (not a multiply by
7/a), round-half-to-even, one scale per token / per output channel, weight
stored [N,K] as in y = x W^T + b, even k in the low nibble, the no-FMA
epilogue order of step 7.

Parity pins live in the CPU tests: hand-worked examples, a rational-arithmetic
quotient check, Python-integer brute force for step 6, closed forms and
invariants.

bf16 values are handled as uint16 bit patterns (numpy has no bf16 type).
"""

import numpy as np

# ---------------------------------------------------------------------------
# bf16 bit helpers
# ---------------------------------------------------------------------------


def bf16_bits_to_f32(bits):
    """bf16 bit patterns (uint16) -> float32, exact (a bf16 is the top half of an fp32)."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_bf16_bits(x):
    """float32 -> bf16 bit patterns, round-to-nearest-even.

    Adds 0x7FFF plus the lowest kept bit, then truncates: the textbook RNE
    for dropping the low 16 bits.  NaN inputs are not expected on this path.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return (r & np.uint64(0xFFFF)).astype(np.uint16)


# ---------------------------------------------------------------------------
# Steps 1-3: per-row symmetric int4 quantiser
# ---------------------------------------------------------------------------

QMIN = -8
QMAX = 7
DENOM = np.float32(7.0)


def row_absmax(x_bits):
    """Step 1: a[m] = max_k |x[m,k]| as float32 (exact)."""
    xf = bf16_bits_to_f32(x_bits)
    return np.max(np.abs(xf), axis=1).astype(np.float32)


def row_scale(absmax):
    """Step 2: s = fl32(a / 7), one IEEE fp32 division per row."""
    a = np.asarray(absmax, dtype=np.float32)
    return (a / DENOM).astype(np.float32)


def quantize_rows(x_bits):
    """Steps 1-3 on a [R, K] bf16 matrix: returns (codes int8 [R,K], scale float32 [R]).

    Each element is divided by its row's scale in fp32 (numpy float32 '/' is
    the IEEE correctly rounded division), rounded half-to-even (np.rint),
    then clamped to [-8, 7].  Rows whose scale is zero get all-zero codes.
    """
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    assert x_bits.ndim == 2
    xf = bf16_bits_to_f32(x_bits)
    s = row_scale(row_absmax(x_bits))
    q = np.zeros(xf.shape, dtype=np.int8)
    nz = s != 0
    if np.any(nz):
        with np.errstate(over="ignore", under="ignore"):
            quot = (xf[nz] / s[nz, None]).astype(np.float32)
        q[nz] = np.clip(np.rint(quot), QMIN, QMAX).astype(np.int8)
    return q, s


# ---------------------------------------------------------------------------
# Step 4: nibble packing
# ---------------------------------------------------------------------------


def pack_int4(q):
    """Pack int codes [R, K] (K even) into bytes [R, K/2]: even k -> low nibble."""
    q = np.asarray(q, dtype=np.int16)
    assert q.ndim == 2 and q.shape[1] % 2 == 0
    lo = q[:, 0::2] & 0xF
    hi = q[:, 1::2] & 0xF
    return (lo | (hi << 4)).astype(np.uint8)


def unpack_int4(packed):
    """Inverse of pack_int4: bytes [R, K/2] -> int8 codes [R, K] (two's complement nibbles)."""
    p = np.asarray(packed, dtype=np.uint8).astype(np.int16)
    lo = p & 0xF
    hi = (p >> 4) & 0xF
    lo = np.where(lo >= 8, lo - 16, lo)
    hi = np.where(hi >= 8, hi - 16, hi)
    out = np.empty((p.shape[0], p.shape[1] * 2), dtype=np.int8)
    out[:, 0::2] = lo
    out[:, 1::2] = hi
    return out


def quantize_act(x_bits):
    """Activation path (steps 1-4): bf16 [M,K] -> (packed uint8 [M,K/2], scale fp32 [M])."""
    q, s = quantize_rows(x_bits)
    return pack_int4(q), s


def pack_weight_int4(w_bits):
    """Weight path (step 5): bf16 W [N,K] -> (packed uint8 [N,K/2], scale fp32 [N]).

    Per-output-channel scaling of an [N,K] weight is per-row scaling.
    """
    q, s = quantize_rows(w_bits)
    return pack_int4(q), s


# ---------------------------------------------------------------------------
# Step 6: exact integer contraction
# ---------------------------------------------------------------------------


def code_gemm(qx, qw):
    """acc[m,n] = sum_k qx[m,k] * qw[n,k], exact, returned as int64 [M,N].

    Computed as a float64 matrix product of the codes: every product and every
    partial sum is an integer of magnitude <= 64*K < 2^53, so the result is
    exact whatever order the library sums in.
    """
    qx = np.asarray(qx)
    qw = np.asarray(qw)
    assert qx.ndim == 2 and qw.ndim == 2 and qx.shape[1] == qw.shape[1]
    assert 64 * qx.shape[1] < 2 ** 53
    acc = qx.astype(np.float64) @ qw.astype(np.float64).T
    return acc.astype(np.int64)


def brute_force_gemm(qx, qw):
    """Python-integer triple loop for tiny shapes (pins code_gemm)."""
    qx = [[int(v) for v in row] for row in np.asarray(qx)]
    qw = [[int(v) for v in row] for row in np.asarray(qw)]
    out = []
    for xr in qx:
        row = []
        for wr in qw:
            t = 0
            for a, b in zip(xr, wr):
                t += a * b
            row.append(t)
        out.append(row)
    return np.array(out, dtype=np.int64).reshape(len(qx), len(qw))


# ---------------------------------------------------------------------------
# Step 7: dequantising epilogue
# ---------------------------------------------------------------------------


def epilogue(acc, s_x, s_w, bias_bits=None):
    """y = bf16_rne(((f32(acc) * s_x[m]) * s_w[n]) + f32(bias[n])), all in fp32.

    numpy evaluates each elementwise float32 operation separately and rounds
    it (no contraction into a fused multiply-add), which is the pinned order.
    f32(acc) is exact because |acc| <= 64*K < 2^24 for K < 262144.
    """
    acc = np.asarray(acc)
    assert np.all(np.abs(acc) < 2 ** 24)
    t = acc.astype(np.float32)
    # rows near the bf16 maximum may overflow to +-inf, the IEEE result
    with np.errstate(over="ignore", invalid="ignore"):
        t = (t * np.asarray(s_x, dtype=np.float32)[:, None]).astype(np.float32)
        t = (t * np.asarray(s_w, dtype=np.float32)[None, :]).astype(np.float32)
        if bias_bits is not None:
            t = (t + bf16_bits_to_f32(bias_bits)[None, :]).astype(np.float32)
    return f32_to_bf16_bits(t)


# ---------------------------------------------------------------------------
# The whole layer
# ---------------------------------------------------------------------------


def w4a4_gemm(qx_packed, s_x, qw_packed, s_w, bias_bits=None):
    """Steps 6-7 on packed operands: returns bf16 bits [M,N]."""
    acc = code_gemm(unpack_int4(qx_packed), unpack_int4(qw_packed))
    return epilogue(acc, s_x, s_w, bias_bits)


def w4a4_gemm_i32(qx_packed, qw_packed):
    """Step 6 only on packed operands: exact accumulators as int32 [M,N]."""
    acc = code_gemm(unpack_int4(qx_packed), unpack_int4(qw_packed))
    return acc.astype(np.int32)


def w4a4_linear(x_bits, qw_packed, s_w, bias_bits=None):
    """Full layer on bf16 activations and a pre-packed weight: bf16 bits [M,N]."""
    qx, s_x = quantize_act(x_bits)
    return w4a4_gemm(qx, s_x, qw_packed, s_w, bias_bits)


def w4a4_linear_rows(x_bits, qw_packed, s_w, rows, bias_bits=None):
    """The layer's output for a subset of rows only (quantisation is row-local).

    Used to check sampled outputs of full-size problems one row at a time.
    """
    rows = np.asarray(rows)
    return w4a4_linear(np.asarray(x_bits)[rows], qw_packed, s_w, bias_bits)
