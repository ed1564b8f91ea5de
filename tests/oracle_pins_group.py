"""Pins for the group-wise W4A4 part of the CPU oracle.

Each pin takes an implementation namespace (an object with quantize_rows_group,
group_code_gemm, group_sum, group_epilogue, pack_int4 and unpack_int4) and
raises AssertionError when it disagrees with what the definition and plain
mathematics fix: a hand-worked example, exact rational arithmetic, Python
integers, the per-token layer it reduces to when one group spans K, and
locality.  The same pins run against the oracle (they must pass) and against
mutants of it (at least one must fail).
"""

from fractions import Fraction

import numpy as np

import oracle
from tests.golden import fixtures
from tests.oracle_pins import bf16_value, exact_bf16_bits, f32_bits, to_bf16, to_f32


def _sparse(K, idx, val):
    row = np.zeros(K, dtype=np.float64)
    row[np.asarray(idx, dtype=np.int64)] = val
    return exact_bf16_bits(row)


def rational_group_row(bits, G):
    """Steps 1-3 in exact rational arithmetic for one row: (codes, scales)."""
    xs = [Fraction(bf16_value(b)) for b in bits]
    q, ss = [], []
    for g in range(len(xs) // G):
        seg = xs[g * G:(g + 1) * G]
        s = to_f32(max(abs(v) for v in seg) / 7)
        ss.append(s)
        q += [0] * G if s == 0 else [max(-8, min(7, round(to_f32(v / s)))) for v in seg]
    return q, ss


def rational_group_sum(acc, sx, sw):
    """Step 7 for one output in exact rational arithmetic with per-operation fp32 rounding."""
    S = Fraction(0)
    for a, x, w in zip(acc, sx, sw):
        t = to_f32(to_f32(Fraction(int(a)) * Fraction(float(x))) * Fraction(float(w)))
        S = to_f32(S + t)
    return S


def pin_golden_group(impl):
    c = fixtures.load("group_examples.txt")["grp_gemm_mini"]
    K, G = c["K"][0], c["G"][0]
    x = _sparse(K, c["x_idx"], c["x_val"])[None, :]
    w0 = exact_bf16_bits(np.repeat(np.array(c["w0_group_vals"], dtype=np.float64), G))
    w1 = _sparse(K, c["w1_idx"], c["w1_val"])
    w = np.stack([w0, w1])
    qx, sx = impl.quantize_rows_group(x, G)
    assert [f32_bits(float(v)) for v in sx[0]] == c["sx_bits"], sx
    nz = np.flatnonzero(qx[0])
    assert nz.tolist() == c["qx_idx"] and qx[0, nz].tolist() == c["qx_val"], qx[0, nz]
    qw, sw = impl.quantize_rows_group(w, G)
    assert [f32_bits(float(v)) for v in sw[0]] == c["sw0_bits"] and np.all(qw[0] == 7)
    assert [f32_bits(float(v)) for v in sw[1]] == c["sw1_bits"]
    assert np.array_equal(impl.unpack_int4(impl.pack_int4(qx)), qx)
    acc = impl.group_code_gemm(qx, qw, G)
    assert acc[0, 0].tolist() == c["acc_n0"] and acc[0, 1].tolist() == c["acc_n1"], acc
    S = impl.group_sum(acc, sx, sw)
    assert [f32_bits(float(v)) for v in S[0]] == c["S_bits"], S
    assert [int(v) for v in impl.group_epilogue(S)[0]] == c["y_bits"]
    assert [int(v) for v in impl.group_epilogue(S, exact_bf16_bits(c["bias"]))[0]] == c["y_bias_bits"]


def pin_rational_group_quantizer(impl, rows, G):
    q, s = impl.quantize_rows_group(rows, G)
    for r in range(rows.shape[0]):
        rq, rs = rational_group_row(rows[r], G)
        assert [Fraction(float(v)) for v in s[r]] == rs, (r, s[r])
        assert q[r].tolist() == rq, r


def pin_rational_group_sum(impl, n=300, ng=6, seed=4):
    rng = np.random.default_rng(seed)
    acc = rng.integers(-8000, 8000, size=(n, 1, ng)).astype(np.int64)
    sx = (rng.uniform(0.5, 2, size=(n, ng)) * 2.0 ** rng.integers(-30, 10, size=(n, ng))).astype(np.float32)
    sw = (rng.uniform(0.5, 2, size=(1, ng)) * 2.0 ** -5).astype(np.float32)
    S = impl.group_sum(acc, sx, sw)
    for i in range(n):
        ref = rational_group_sum(acc[i, 0], sx[i], sw[0])
        assert Fraction(float(S[i, 0])) == ref, (i, S[i, 0], float(ref))


def pin_group_epilogue_rational(impl, n=200, seed=6):
    rng = np.random.default_rng(seed)
    S = (rng.standard_normal((1, n)) * 10.0 ** rng.integers(-3, 4, size=(1, n))).astype(np.float32)
    b = exact_bf16_bits(np.round(rng.standard_normal(n) * 64) / 64)
    y = impl.group_epilogue(S, b)
    for j in range(n):
        ref = to_bf16(to_f32(Fraction(float(S[0, j])) + Fraction(bf16_value(b[j]))))
        assert Fraction(bf16_value(y[0, j])) == ref, j


def pin_group_brute_force(impl, G, seed=8):
    rng = np.random.default_rng(seed)
    M, N, K = 3, 4, 2 * G
    qx = rng.integers(-8, 8, size=(M, K)).astype(np.int8)
    qw = rng.integers(-8, 8, size=(N, K)).astype(np.int8)
    acc = impl.group_code_gemm(qx, qw, G)
    for m in range(M):
        for n in range(N):
            for g in range(K // G):
                want = sum(int(qx[m, k]) * int(qw[n, k]) for k in range(g * G, (g + 1) * G))
                assert acc[m, n, g] == want, (m, n, g)


def pin_reduces_to_per_token(impl, x_bits, w_bits, b_bits):
    """With one group spanning K the layer is the per-token W4A4 layer (itself pinned separately)."""
    K = x_bits.shape[1]
    qx, sx = impl.quantize_rows_group(x_bits, K)
    qw, sw = impl.quantize_rows_group(w_bits, K)
    y = impl.group_epilogue(impl.group_sum(impl.group_code_gemm(qx, qw, K), sx, sw), b_bits)
    pq, ps = oracle.quantize_rows(x_bits)
    assert np.array_equal(qx, pq) and np.array_equal(sx[:, 0], ps)
    wq, ws = oracle.pack_weight_int4(w_bits)
    assert np.array_equal(y, oracle.w4a4_gemm(oracle.pack_int4(pq), ps, wq, ws, b_bits))


def pin_group_locality(impl, rows, G):
    """Changing one group of a row changes only that group's codes and scale."""
    q, s = impl.quantize_rows_group(rows, G)
    ng = rows.shape[1] // G
    for g in range(ng):
        r2 = rows.copy()
        r2[:, g * G:(g + 1) * G] = r2[:, g * G:(g + 1) * G][:, ::-1]  # reorder inside the group
        q2, s2 = impl.quantize_rows_group(r2, G)
        keep = np.ones(rows.shape[1], bool)
        keep[g * G:(g + 1) * G] = False
        assert np.array_equal(q2[:, keep], q[:, keep])
        assert np.array_equal(np.delete(s2, g, axis=1), np.delete(s, g, axis=1))
        assert np.array_equal(s2[:, g], s[:, g])  # a reorder keeps the group's absmax
        assert np.array_equal(q2[:, g * G:(g + 1) * G], q[:, g * G:(g + 1) * G][:, ::-1])


def pin_group_invariants(impl, rows, G):
    q, s = impl.quantize_rows_group(rows, G)
    assert q.min() >= -8 and q.max() <= 7
    x = (rows.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    sg = np.repeat(s.astype(np.float64), G, axis=1)
    assert np.all(np.abs(x - q * sg) <= 0.5 * sg * (1 + 2.0 ** -20))
    # the absmax element of every nonzero group maps to +-7
    xg = np.abs(x).reshape(x.shape[0], -1, G)
    qg = np.abs(q).reshape(q.shape[0], -1, G)
    arg = np.argmax(xg, axis=2)
    top = np.take_along_axis(qg, arg[:, :, None], axis=2)[:, :, 0]
    assert np.all(top[s > 0] == 7)
