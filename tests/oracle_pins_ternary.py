"""Pins for the ternary (W1.58A4) part of the CPU oracle.

Each pin takes an implementation namespace (an object with quantize_ternary,
pack_ternary, unpack_ternary, quantize_act, code_gemm, unpack_int4 and
epilogue) and raises AssertionError when it disagrees with what the definition
and plain mathematics fix: hand-worked examples, exact rational arithmetic,
bit-by-bit packing, closed forms and symmetries.  The same pins run against the
oracle (they must pass) and against mutants of it (at least one must fail).
"""

from fractions import Fraction

import numpy as np

from tests.golden import fixtures
from tests.oracle_pins import bf16_value, exact_bf16_bits, f32_bits, to_f32


def rational_ternary_row(bits):
    """Steps 1-2 of the ternary quantiser in exact rational arithmetic for one row.

    The sum of |w| is exact (Fraction); its quotient by K is rounded to the
    nearest float64 (Python float of a Fraction is correctly rounded), then to
    float32; each code is the RNE of the correctly rounded fp32 quotient.
    """
    ws = [Fraction(bf16_value(b)) for b in bits]
    S = sum(abs(v) for v in ws)
    g = to_f32(Fraction(float(S / len(ws))))
    if g == 0:
        return [0] * len(ws), g
    t = [max(-1, min(1, round(to_f32(v / g)))) for v in ws]
    return t, g


def pin_golden_ternary(impl):
    cases = fixtures.load("ternary_examples.txt")
    for name in ("tern1_basic", "tern2_ties", "tern3_zero_row", "tern4_clamp_negative"):
        c = cases[name]
        w = exact_bf16_bits(c["w"])[None, :]
        t, g = impl.quantize_ternary(w)
        assert list(t[0]) == c["t"], (name, list(t[0]))
        assert f32_bits(float(g[0])) == c["g_bits"][0], (name, g[0])
        assert list(impl.pack_ternary(t)[0]) == c["packed"], name


def pin_golden_ternary_gemm(impl):
    cases = fixtures.load("ternary_examples.txt")
    c = cases["tern_gemm_mini"]
    x = exact_bf16_bits(c["x"])[None, :]
    w = np.stack([exact_bf16_bits(cases["tern1_basic"]["w"]), exact_bf16_bits(cases["tern2_ties"]["w"])])
    qx, sx = impl.quantize_act(x)
    t, g = impl.quantize_ternary(w)
    acc = impl.code_gemm(impl.unpack_int4(qx), impl.unpack_ternary(impl.pack_ternary(t)))
    assert list(acc[0]) == c["acc"], acc
    y = impl.epilogue(acc, sx, g)
    assert [int(v) for v in y[0]] == c["y_bits"], [hex(v) for v in y[0]]
    yb = impl.epilogue(acc, sx, g, exact_bf16_bits(c["bias"]))
    assert [int(v) for v in yb[0]] == c["y_bias_bits"], [hex(v) for v in yb[0]]


def pin_rational_ternary(impl, rows):
    t, g = impl.quantize_ternary(rows)
    for r in range(rows.shape[0]):
        tr, gr = rational_ternary_row(rows[r])
        assert Fraction(float(g[r])) == gr, (r, g[r], gr)
        assert list(t[r]) == tr, (r, list(t[r]), tr)


def pin_ternary_pack_bits(impl, t):
    """Bit-by-bit construction of the 2-bit fields, and the round trip."""
    p = impl.pack_ternary(t)
    assert p.shape == (t.shape[0], t.shape[1] // 4) and p.dtype == np.uint8
    for r in range(t.shape[0]):
        for j in range(t.shape[1] // 4):
            byte = 0
            for i in range(4):
                v = int(t[r, 4 * j + i])
                field = {0: 0b00, 1: 0b01, -1: 0b11}[v]
                byte |= field << (2 * i)
            assert int(p[r, j]) == byte, (r, j, hex(int(p[r, j])), hex(byte))
    assert np.array_equal(impl.unpack_ternary(p), t)


def pin_ternary_closed_forms(impl):
    K = 64
    # constant-magnitude rows: g = |c| and t = sign(w)
    for c in (1.0, 0.375, 2.0 ** -20, 96.0):
        rng = np.random.default_rng(int(c * 1e6) % 1000)
        signs = rng.choice([-1.0, 1.0], size=K)
        w = exact_bf16_bits(signs * c)[None, :]
        t, g = impl.quantize_ternary(w)
        assert float(g[0]) == c, (c, g)
        assert np.array_equal(t[0], signs.astype(np.int8))
    # one nonzero element: g = |w|/K, the element saturates to +-1, the rest are 0
    w = np.zeros((1, K), dtype=np.uint16)
    w[0, 7] = exact_bf16_bits([-3.0])[0]
    t, g = impl.quantize_ternary(w)
    assert float(g[0]) == 3.0 / K
    assert t[0, 7] == -1 and np.count_nonzero(t) == 1


def pin_ternary_symmetries(impl, rows):
    t, g = impl.quantize_ternary(rows)
    # sign flip: same scale, negated codes
    tn, gn = impl.quantize_ternary(rows ^ np.uint16(0x8000))
    assert np.array_equal(gn, g) and np.array_equal(tn, -t)
    # power-of-two scaling: bf16 exponent + 2 scales w by 4, g by 4, codes unchanged
    # (rows must hold normal numbers or zeros only)
    nz = (rows & 0x7FFF) != 0
    assert np.all((rows[nz] & 0x7F80) != 0), "subnormal input"
    assert np.all((rows[nz] & 0x7F80) < 0x7C00)
    up = rows.copy()
    up[nz] = rows[nz] + np.uint16(2 << 7)
    tu, gu = impl.quantize_ternary(up)
    assert np.array_equal(tu, t) and np.array_equal(gu, (g * np.float32(4)).astype(np.float32))
    # row permutation within K does not change the scale (the sum is exact)
    perm = np.random.default_rng(3).permutation(rows.shape[1])
    tp, gp = impl.quantize_ternary(rows[:, perm])
    assert np.array_equal(gp, g) and np.array_equal(tp, t[:, perm])


def pin_ternary_invariants(impl, rows):
    """Codes lie in {-1, 0, 1}; where |w| < 1.5 g (no clamping) the error is at most g/2."""
    t, g = impl.quantize_ternary(rows)
    assert set(np.unique(t)).issubset({-1, 0, 1})
    w = (rows.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    gg = g.astype(np.float64)[:, None]
    inside = np.abs(w) < 1.5 * gg * (1 - 2.0 ** -20)
    err = np.abs(w - t * gg)
    assert np.all(err[inside] <= 0.5 * gg.repeat(w.shape[1], 1)[inside] * (1 + 2.0 ** -20))
    # clamped elements carry the sign of w
    outside = np.abs(w) >= 1.5 * gg * (1 + 2.0 ** -20)
    assert np.all(t[outside] == np.sign(w[outside]))
