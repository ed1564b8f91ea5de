"""Pins for the CPU oracle: checks that fix the oracle to something other than itself.

Each pin takes an implementation namespace (an object with quantize_rows,
pack_int4, unpack_int4, code_gemm and epilogue) and raises AssertionError when
the implementation disagrees with what the paper's operator and plain
mathematics fix: hand-worked examples, exact rational arithmetic, Python-integer
brute force, closed forms and invariants.  The same pins run against the
oracle (they must pass) and against mutants of it that carry a plausible
mistake (at least one pin must fail), which shows the pins have teeth.
"""

import struct
from fractions import Fraction

import numpy as np

from tests.golden import fixtures

# ---------------------------------------------------------------------------
# helpers that do not use the oracle
# ---------------------------------------------------------------------------


def f32_bits(v):
    return struct.unpack("<I", struct.pack("<f", v))[0]


def bits_f32(b):
    return struct.unpack("<f", struct.pack("<I", b))[0]


def exact_bf16_bits(vals):
    """Bit patterns of values that are exactly representable in bf16."""
    out = []
    for v in vals:
        b = f32_bits(float(v))
        assert b & 0xFFFF == 0, f"{v} is not a bf16 value"
        out.append(b >> 16)
    return np.array(out, dtype=np.uint16)


def bf16_value(b):
    return bits_f32(int(b) << 16)


def round_fraction(r, mant_bits, min_exp):
    """Round a rational to the nearest binary float with `mant_bits` fraction
    bits and smallest quantum 2**min_exp, ties to even (IEEE RNE)."""
    if r == 0:
        return Fraction(0)
    sign = -1 if r < 0 else 1
    a = abs(r)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    quantum = Fraction(2) ** max(e - mant_bits, min_exp)
    return sign * round(a / quantum) * quantum


def to_f32(r):
    return round_fraction(r, 23, -149)


def to_bf16(r):
    return round_fraction(r, 7, -133)


def rational_quantize_row(bits):
    """Steps 1-3 of the quantiser in exact rational arithmetic for one row."""
    xs = [Fraction(bf16_value(b)) for b in bits]
    a = max(abs(v) for v in xs)
    s = to_f32(a / 7)
    if s == 0:
        return [0] * len(xs), s
    q = [max(-8, min(7, round(to_f32(v / s)))) for v in xs]
    return q, s


# ---------------------------------------------------------------------------
# pins
# ---------------------------------------------------------------------------


def pin_golden_quantizer(impl):
    cases = fixtures.load("quantizer_examples.txt")
    for name in ("ex1_ties", "ex2_division_not_reciprocal", "ex3_zero_row", "ex4_negative_max"):
        c = cases[name]
        x = exact_bf16_bits(c["x"])[None, :]
        q, s = impl.quantize_rows(x)
        assert list(np.asarray(q[0], dtype=int)) == c["q"], (name, q[0], c["q"])
        assert f32_bits(float(s[0])) == c["s_bits"][0], (name, hex(f32_bits(float(s[0]))))
        packed = impl.pack_int4(q)
        assert list(np.asarray(packed[0], dtype=int)) == c["packed"], (name, packed[0])
        back = impl.unpack_int4(packed)
        assert np.array_equal(back, np.asarray(q, dtype=np.int8)), name


def pin_golden_gemm(impl):
    c = fixtures.load("quantizer_examples.txt")["gemm_mini"]
    x = exact_bf16_bits(c["x"])[None, :]
    w = np.stack([exact_bf16_bits(c["w0"]), exact_bf16_bits(c["w1"])])
    qx, sx = impl.quantize_rows(x)
    qw, sw = impl.quantize_rows(w)
    assert list(np.asarray(qw[0], dtype=int)) == c["qw0"]
    assert list(np.asarray(qw[1], dtype=int)) == c["qw1"]
    assert [f32_bits(float(v)) for v in sw] == c["sw_bits"]
    acc = impl.code_gemm(qx, qw)
    assert list(np.asarray(acc[0], dtype=int)) == c["acc"], acc
    y = impl.epilogue(acc, sx, sw, None)
    assert list(np.asarray(y[0], dtype=int)) == c["y_bits"], [hex(v) for v in y[0]]
    b = exact_bf16_bits(c["bias"])
    yb = impl.epilogue(acc, sx, sw, b)
    assert list(np.asarray(yb[0], dtype=int)) == c["y_bias_bits"], [hex(v) for v in yb[0]]


def pin_rational_quantizer(impl, rows):
    """Quotient, rounding and clamp against exact rational arithmetic."""
    q, s = impl.quantize_rows(rows)
    for r in range(rows.shape[0]):
        rq, rs = rational_quantize_row(rows[r])
        assert Fraction(float(s[r])) == rs, (r, float(s[r]), float(rs))
        assert list(np.asarray(q[r], dtype=int)) == rq, r


def brute_force_dot(qx, qw):
    """acc[m][n] = sum_k qx[m][k] * qw[n][k] with Python integers."""
    xs = [[int(v) for v in row] for row in np.asarray(qx)]
    ws = [[int(v) for v in row] for row in np.asarray(qw)]
    return np.array([[sum(a * b for a, b in zip(xr, wr)) for wr in ws] for xr in xs],
                    dtype=np.int64).reshape(len(xs), len(ws))


def pin_brute_force_gemm(impl, qx, qw):
    got = np.asarray(impl.code_gemm(qx, qw), dtype=np.int64)
    exp = brute_force_dot(qx, qw)
    assert got.shape == exp.shape, (got.shape, exp.shape)
    assert np.array_equal(got, exp)


def pin_extreme_accumulators(impl, K):
    """Codes all at the same extreme: acc = -49K, -56K, 56K, 64K in closed form."""
    qx = np.full((2, K), 7, np.int8)
    qx[1] = -8
    qw = np.full((2, K), -7, np.int8)
    qw[1] = -8
    acc = np.asarray(impl.code_gemm(qx, qw), dtype=np.int64)
    assert acc.tolist() == [[-49 * K, -56 * K], [56 * K, 64 * K]], acc


def pin_epilogue_rational(impl, acc, sx, sw, bias_bits, samples):
    """Epilogue against per-operation rational rounding, on sampled elements."""
    y = impl.epilogue(acc, sx, sw, bias_bits)
    for m, n in samples:
        t = to_f32(Fraction(int(acc[m, n])))
        t = to_f32(t * Fraction(float(sx[m])))
        t = to_f32(t * Fraction(float(sw[n])))
        if bias_bits is not None:
            t = to_f32(t + Fraction(bf16_value(bias_bits[n])))
        exp = to_bf16(t)
        got = Fraction(bf16_value(y[m, n]))
        assert got == exp, (m, n, float(got), float(exp))


def pin_epilogue_fp64(impl, acc, sx, sw, bias_bits):
    """Epilogue on many elements against an fp64 emulation of each fp32 operation.

    A product of two fp32 values is exact in fp64, and for a sum of two fp32
    values rounding first to fp64 and then to fp32 equals a single rounding
    (53 >= 2*24 + 2), so casting each fp64 result to fp32 reproduces IEEE fp32
    arithmetic operation by operation.  The final bf16 rounding is torch's cast.
    """
    import torch

    y = impl.epilogue(acc, sx, sw, bias_bits)
    t = np.asarray(acc, dtype=np.float64).astype(np.float32).astype(np.float64)
    t = (t * np.asarray(sx, np.float32).astype(np.float64)[:, None]).astype(np.float32)
    t = (t.astype(np.float64) * np.asarray(sw, np.float32).astype(np.float64)[None, :]).astype(np.float32)
    if bias_bits is not None:
        b = np.array([bf16_value(v) for v in bias_bits], dtype=np.float64)
        t = (t.astype(np.float64) + b[None, :]).astype(np.float32)
    ref = torch.from_numpy(t).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    bad = np.argwhere(np.asarray(y) != ref)
    assert bad.size == 0, (len(bad), bad[:3])


def pin_invariants(impl, rows):
    q, s = impl.quantize_rows(rows)
    q = np.asarray(q, dtype=np.int64)
    xf = np.array([[bf16_value(b) for b in r] for r in rows], dtype=np.float64)
    assert q.min() >= -8 and q.max() <= 7
    for r in range(rows.shape[0]):
        a = np.max(np.abs(xf[r]))
        if a == 0:
            assert s[r] == 0 and np.all(q[r] == 0)
            continue
        k = int(np.argmax(np.abs(xf[r])))
        assert abs(q[r, k]) == 7 and np.sign(q[r, k]) == np.sign(xf[r, k]), r
        err = np.abs(xf[r] - q[r] * np.float64(s[r]))
        assert np.all(err <= np.float64(s[r]) / 2 * (1 + 2.0 ** -20)), (r, err.max() / s[r])
    packed = impl.pack_int4(q)
    assert packed.shape == (rows.shape[0], rows.shape[1] // 2)
    assert np.array_equal(impl.unpack_int4(packed), q.astype(np.int8))


def pin_scale_equivariance(impl, rows):
    """Multiplying a row by 2^e (no over/underflow) scales s by 2^e and keeps q."""
    q, s = impl.quantize_rows(rows)
    xf = np.array([[bf16_value(b) for b in r] for r in rows], dtype=np.float32)
    for e in (-3, 5):
        xs = (xf * np.float32(2.0 ** e)).astype(np.float32)
        bits = (xs.view(np.uint32) >> 16).astype(np.uint16)
        q2, s2 = impl.quantize_rows(bits)
        assert np.array_equal(np.asarray(q2), np.asarray(q))
        assert np.array_equal(np.asarray(s2, dtype=np.float32),
                              (np.asarray(s, dtype=np.float32) * np.float32(2.0 ** e)))


def pin_closed_forms(impl):
    # constant magnitude rows -> all codes +-7
    rng = np.random.default_rng(7)
    signs = rng.choice([-1.0, 1.0], size=(4, 32))
    mags = np.array([0.75, 3.0, 1.0 / 1024, 96.0])[:, None]
    q, _ = impl.quantize_rows(exact_bf16_bits((signs * mags).ravel()).reshape(4, 32))
    assert np.array_equal(np.asarray(q, dtype=np.int64), (7 * signs).astype(np.int64))
    # integer rows k * 2^e with max |k| = 7 -> q = k, s = 2^e
    k = rng.integers(-7, 8, size=(6, 32))
    k[:, 3] = np.array([7, -7, 7, -7, 7, -7])
    ex = np.array([0, -4, 3, -9, 10, -1])
    vals = k * (2.0 ** ex)[:, None]
    q, s = impl.quantize_rows(exact_bf16_bits(vals.ravel()).reshape(k.shape))
    assert np.array_equal(np.asarray(q, dtype=np.int64), k)
    assert np.array_equal(np.asarray(s, dtype=np.float64), 2.0 ** ex)
    # W = c*I: each weight row has one non-zero, so qW = 7 I and acc = 7 qX
    K = 64
    x = exact_bf16_bits(rng.integers(-40, 41, size=(5, K)).ravel() / 8.0).reshape(5, K)
    w = exact_bf16_bits((0.375 * np.eye(K)).ravel()).reshape(K, K)
    qx, _ = impl.quantize_rows(x)
    qw, sw = impl.quantize_rows(w)
    assert np.array_equal(np.asarray(qw, dtype=np.int64), 7 * np.eye(K, dtype=np.int64))
    assert np.all(np.asarray(sw, dtype=np.float32) == np.float32(np.float32(0.375) / np.float32(7)))
    acc = impl.code_gemm(qx, qw)
    assert np.array_equal(np.asarray(acc, dtype=np.int64), 7 * np.asarray(qx, dtype=np.int64))


def pin_permutation_invariance(impl, qx, qw):
    perm = np.random.default_rng(3).permutation(qx.shape[1])
    a = impl.code_gemm(qx, qw)
    b = impl.code_gemm(qx[:, perm], qw[:, perm])
    assert np.array_equal(np.asarray(a), np.asarray(b))


def pin_sanity_bound(impl, x_bits, w_bits, bias_bits=None):
    """|y - x W^T - b| stays within the quantisation error bound plus bf16 rounding."""
    qx, sx = impl.quantize_rows(x_bits)
    qw, sw = impl.quantize_rows(w_bits)
    acc = impl.code_gemm(qx, qw)
    y = impl.epilogue(acc, sx, sw, bias_bits)
    xf = np.array([[bf16_value(b) for b in r] for r in x_bits], dtype=np.float64)
    wf = np.array([[bf16_value(b) for b in r] for r in w_bits], dtype=np.float64)
    ref = xf @ wf.T
    if bias_bits is not None:
        ref = ref + np.array([bf16_value(b) for b in bias_bits])[None, :]
    sxd = np.asarray(sx, dtype=np.float64)[:, None]
    swd = np.asarray(sw, dtype=np.float64)[None, :]
    bound = (np.abs(xf).sum(1)[:, None] * swd / 2 + np.abs(wf).sum(1)[None, :] * sxd / 2
             + xf.shape[1] * sxd * swd / 4) * (1 + 1e-5)
    yv = np.array([[bf16_value(b) for b in r] for r in y], dtype=np.float64)
    assert np.all(np.abs(yv - ref) <= bound + np.abs(ref + bound) * 2.0 ** -8 + 1e-30)


ALL_PINS = (
    "pin_golden_quantizer",
    "pin_golden_gemm",
    "pin_rational_quantizer",
    "pin_brute_force_gemm",
    "pin_epilogue_rational",
    "pin_invariants",
    "pin_scale_equivariance",
    "pin_closed_forms",
    "pin_permutation_invariance",
)
