"""The ternary (W1.58A4) part of the CPU oracle against its pins (no GPU needed).

Mutant tests plant plausible mistakes in copies of the oracle, on the CPU, and
check that at least one pin catches each of them.
"""

import types

import numpy as np
import pytest

import oracle
from paper_2609_33601_amd import workloads
from tests import oracle_pins_ternary as PT
from tests.oracle_pins import exact_bf16_bits


def _tie_rows(n_rows=16, K=32, seed=5):
    """Rows with elements exactly at w/g = +-0.5 and +-1.5 (the decision points).

    The block 6 4.5 1.5 1.5 3 4.5 3 0 sums to 24 over 8 elements, so g = 3 and
    the 1.5s sit at w/g = 0.5, the 4.5s at 1.5.  Tiled to K, scaled by a power
    of two, with random signs and order, the scale stays g = 3 * 2^j.
    """
    rng = np.random.default_rng(seed)
    base = np.array([6, 4.5, 1.5, 1.5, 3, 4.5, 3, 0], dtype=np.float64)
    rows = []
    for _ in range(n_rows):
        row = np.tile(base, K // 8) * (2.0 ** rng.integers(-12, 12))
        row *= rng.choice([-1.0, 1.0], size=K)
        rows.append(exact_bf16_bits(row[rng.permutation(K)]))
    return np.stack(rows)


def _random_rows(n=24, K=256, seed=9):
    rng = np.random.default_rng(seed)
    w = (rng.standard_normal((n, K)) * 0.02).astype(np.float32)
    w[3] = 0.0
    w[5, :] = 0.0
    w[5, 17] = 0.5
    bits = (w.view(np.uint32) + np.uint32(0x7FFF) + ((w.view(np.uint32) >> 16) & 1)) >> np.uint32(16)
    return bits.astype(np.uint16)


def _workload_rows():
    return workloads.weights(8, 512, 0.02, 7)


def _normal_only(rows):
    r = rows.copy()
    sub = ((r & 0x7F80) == 0) & ((r & 0x7F) != 0)
    r[sub] = 0
    return r


def _run_pins(impl):
    PT.pin_golden_ternary(impl)
    PT.pin_golden_ternary_gemm(impl)
    rows = np.concatenate([_tie_rows(), _random_rows()[:, :32]])
    PT.pin_rational_ternary(impl, rows)
    PT.pin_rational_ternary(impl, _workload_rows()[:, :128])
    rng = np.random.default_rng(2)
    PT.pin_ternary_pack_bits(impl, rng.integers(-1, 2, size=(6, 64)).astype(np.int8))
    PT.pin_ternary_closed_forms(impl)
    PT.pin_ternary_symmetries(impl, _normal_only(np.concatenate([_random_rows(), _workload_rows()[:, :256]])))
    PT.pin_ternary_invariants(impl, np.concatenate([_random_rows(), _workload_rows()[:, :256]]))


def test_pins_pass_on_oracle():
    _run_pins(oracle)


def test_tie_rows_hit_the_decision_points():
    t, g = oracle.quantize_ternary(_tie_rows())
    w = (_tie_rows().astype(np.uint32) << 16).view(np.float32)
    q = np.abs(w / g[:, None])
    assert np.any(q == 0.5) and np.any(q == 1.5)


def test_brute_force_ternary_gemm():
    rng = np.random.default_rng(4)
    for (M, N, K) in ((1, 1, 4), (3, 5, 8), (7, 4, 64), (8, 8, 128)):
        qx = rng.integers(-8, 8, size=(M, K)).astype(np.int8)
        t = rng.integers(-1, 2, size=(N, K)).astype(np.int8)
        packed_x = oracle.pack_int4(qx)
        packed_t = oracle.pack_ternary(t)
        want = np.array([[sum(int(a) * int(b) for a, b in zip(qx[m], t[n])) for n in range(N)] for m in range(M)])
        assert np.array_equal(oracle.w158a4_gemm_i32(packed_x, packed_t), want)


def test_extreme_ternary_accumulators():
    K = 65536
    qx = np.full((2, K), -8, dtype=np.int8)
    qx[1] = 7
    t = np.full((2, K), -1, dtype=np.int8)
    t[1] = 1
    acc = oracle.w158a4_gemm_i32(oracle.pack_int4(qx), oracle.pack_ternary(t))
    assert acc.tolist() == [[8 * K, -8 * K], [-7 * K, 7 * K]]


def test_layer_composition():
    lin = workloads.WORKLOADS["tiny"].linears[0]
    x = lin.make_x()
    w = lin.make_w()
    packed, g = oracle.pack_weight_ternary(w)
    y = oracle.w158a4_linear(x, packed, g)
    qx, sx = oracle.quantize_act(x)
    acc = oracle.code_gemm(oracle.unpack_int4(qx), oracle.unpack_ternary(packed))
    assert np.array_equal(y, oracle.epilogue(acc, sx, g))
    rows = np.array([0, 5, 63])
    assert np.array_equal(oracle.w158a4_linear_rows(x, packed, g, rows), y[rows])


# ---------------------------------------------------------------------------
# mutants
# ---------------------------------------------------------------------------


def _ns(**over):
    base = {n: getattr(oracle, n) for n in ("quantize_ternary", "pack_ternary", "unpack_ternary", "quantize_act",
                                            "code_gemm", "unpack_int4", "epilogue")}
    base.update(over)
    return types.SimpleNamespace(**base)


def _qt_variant(scale="absmean", rounding="rne", lo=-1, hi=1, per_tensor=False):
    def quantize_ternary(w_bits):
        wf = oracle.bf16_bits_to_f32(w_bits)
        a = np.abs(wf.astype(np.float64))
        if scale == "absmean":
            S = a.sum(axis=1) if not per_tensor else np.full(a.shape[0], a.sum() / a.shape[0])
            g = (S / a.shape[1]).astype(np.float32)
        elif scale == "absmax":
            g = a.max(axis=1).astype(np.float32)
        elif scale == "mean_f32":
            g = (np.abs(wf).sum(axis=1, dtype=np.float32) / np.float32(a.shape[1])).astype(np.float32)
        t = np.zeros(wf.shape, dtype=np.int8)
        nz = g != 0
        quot = (wf[nz] / g[nz, None]).astype(np.float32)
        if rounding == "rne":
            r = np.rint(quot)
        elif rounding == "away":
            r = np.sign(quot) * np.floor(np.abs(quot) + 0.5)
        elif rounding == "trunc":
            r = np.trunc(quot)
        t[nz] = np.clip(r, lo, hi).astype(np.int8)
        return t, g
    return quantize_ternary


def _pack_reversed(t):
    t = np.asarray(t, dtype=np.int16)
    out = np.zeros((t.shape[0], t.shape[1] // 4), dtype=np.int16)
    for i in range(4):
        out |= (t[:, i::4] & 0x3) << (6 - 2 * i)
    return out.astype(np.uint8)


def _unpack_reversed(p):
    p = np.asarray(p, dtype=np.uint8).astype(np.int16)
    out = np.empty((p.shape[0], p.shape[1] * 4), dtype=np.int8)
    for i in range(4):
        f = (p >> (6 - 2 * i)) & 0x3
        out[:, i::4] = np.where(f >= 2, f - 4, f)
    return out


def _pack_biased(t):
    t = np.asarray(t, dtype=np.int16) + 1
    out = np.zeros((t.shape[0], t.shape[1] // 4), dtype=np.int16)
    for i in range(4):
        out |= (t[:, i::4] & 0x3) << (2 * i)
    return out.astype(np.uint8)


def _unpack_biased(p):
    p = np.asarray(p, dtype=np.uint8).astype(np.int16)
    out = np.empty((p.shape[0], p.shape[1] * 4), dtype=np.int8)
    for i in range(4):
        out[:, i::4] = ((p >> (2 * i)) & 0x3) - 1
    return out


MUTANTS = {
    "absmax_scale": _ns(quantize_ternary=_qt_variant(scale="absmax")),
    "per_tensor_scale": _ns(quantize_ternary=_qt_variant(per_tensor=True)),
    "round_half_away": _ns(quantize_ternary=_qt_variant(rounding="away")),
    "truncate": _ns(quantize_ternary=_qt_variant(rounding="trunc")),
    "clamp_two_bit_range": _ns(quantize_ternary=_qt_variant(lo=-2, hi=1)),
    "reversed_fields": _ns(pack_ternary=_pack_reversed, unpack_ternary=_unpack_reversed),
    "biased_encoding": _ns(pack_ternary=_pack_biased, unpack_ternary=_unpack_biased),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    with pytest.raises(AssertionError):
        _run_pins(MUTANTS[name])
