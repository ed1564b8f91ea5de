"""The CPU oracle against its pins (no GPU needed).

Each pin fixes the oracle to something other than itself (see oracle_pins.py).
The mutant tests plant plausible mistakes in copies of the oracle, on the CPU,
and check that at least one pin catches each of them.
"""

import types

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
from paper_2609_33601_amd import workloads
from tests import oracle_pins as P

# ---------------------------------------------------------------------------
# inputs
# ---------------------------------------------------------------------------


def _near_tie_rows(n_rows=24, K=32, seed=11):
    """Rows whose elements sit next to the half-integer decision points x/s = k + 1/2."""
    rng = np.random.default_rng(seed)
    rows = []
    for _ in range(n_rows):
        a = np.float32(2.0 ** rng.integers(-20, 20) * rng.uniform(1, 2))
        s = np.float64(a) / 7.0
        ks = rng.integers(-7, 7, size=K) + 0.5
        vals = (ks * s).astype(np.float32)
        vals[0] = a
        bits = (vals.view(np.uint32) + np.uint32(0x8000)) >> np.uint32(16)
        # nudge by one bf16 ulp either way to land on both sides of the tie
        bits = bits.astype(np.int64) + rng.integers(-1, 2, size=K)
        bits[0] = np.float32(a).view(np.uint32) >> 16
        rows.append(bits.astype(np.uint16))
    return np.stack(rows)


def _workload_rows():
    w = workloads.WORKLOADS["tiny"].linears[0]
    x = w.make_x()[:8, :64]
    heavy = workloads.activations(8, 64, "student_t3", 5, 0.05, 50.0)
    gelu = workloads.activations(8, 64, "gelu_normal", 6, 0.05, 30.0)
    tiny = np.full((2, 64), 0x0003, dtype=np.uint16)  # bf16 subnormals
    tiny[1, 5] = 0x8001
    return np.concatenate([x, heavy, gelu, tiny])


def _codes(M, N, K, seed):
    rng = np.random.default_rng(seed)
    return (rng.integers(-7, 8, size=(M, K)).astype(np.int8),
            rng.integers(-7, 8, size=(N, K)).astype(np.int8))


# ---------------------------------------------------------------------------
# the oracle passes every pin
# ---------------------------------------------------------------------------


def test_golden_quantizer_examples():
    P.pin_golden_quantizer(oracle)


def test_golden_gemm_example():
    P.pin_golden_gemm(oracle)


def test_quotient_against_rational_arithmetic():
    P.pin_rational_quantizer(oracle, _workload_rows())
    P.pin_rational_quantizer(oracle, _near_tie_rows())


def test_brute_force_tiny_workload():
    """Python-integer dot products on the whole 64x256 -> 256 workload."""
    lin = workloads.WORKLOADS["tiny"].linears[0]
    qx, _ = oracle.quantize_rows(lin.make_x())
    qw, _ = oracle.quantize_rows(lin.make_w())
    P.pin_brute_force_gemm(oracle, qx, qw)


@pytest.mark.parametrize("M,N,K", [(1, 1, 2), (3, 5, 16), (8, 2, 128), (5, 8, 70)])
def test_brute_force_random_shapes(M, N, K):
    qx, qw = _codes(M, N, K, seed=M * 100 + N * 10 + K)
    P.pin_brute_force_gemm(oracle, qx, qw)


def test_code_gemm_matches_int64_matmul():
    qx, qw = _codes(96, 80, 3072, seed=4)
    ref = qx.astype(np.int64) @ qw.astype(np.int64).T
    assert np.array_equal(oracle.code_gemm(qx, qw), ref)


def test_extreme_accumulators_exact():
    """All codes at the same extreme: acc = +-49K and 64K exactly at K = 12288."""
    P.pin_extreme_accumulators(oracle, 12288)


def test_epilogue_against_rational_rounding():
    rng = np.random.default_rng(9)
    acc = rng.integers(-300000, 300000, size=(6, 7)).astype(np.int64)
    acc[0, 0] = 0
    sx = (rng.uniform(0.01, 3, size=6)).astype(np.float32)
    sw = (rng.uniform(1e-4, 1e-2, size=7)).astype(np.float32)
    b = workloads.bias(7, 0.01, 2)
    samples = [(m, n) for m in range(6) for n in range(7)]
    P.pin_epilogue_rational(oracle, acc, sx, sw, None, samples)
    P.pin_epilogue_rational(oracle, acc, sx, sw, b, samples)


def _epilogue_stress(M=1000, N=2000, seed=13):
    rng = np.random.default_rng(seed)
    acc = rng.integers(-600000, 600000, size=(M, N)).astype(np.int64)
    sx = rng.uniform(0.01, 3, size=M).astype(np.float32)
    sw = rng.uniform(1e-4, 1e-2, size=N).astype(np.float32)
    b = workloads.bias(N, 0.05, 14)
    return acc, sx, sw, b


def test_epilogue_against_fp64_emulation():
    acc, sx, sw, b = _epilogue_stress()
    P.pin_epilogue_fp64(oracle, acc, sx, sw, b)
    P.pin_epilogue_fp64(oracle, acc, sx, sw, None)


def test_bf16_rounding_matches_torch_cast():
    import torch

    rng = np.random.default_rng(12)
    u = rng.integers(0, 2 ** 32, size=200000, dtype=np.uint64).astype(np.uint32)
    u = u[((u >> 23) & 0xFF) != 0xFF]  # finite only
    ties = (u & np.uint32(0xFFFF0000)) | np.uint32(0x8000)  # exact halfway cases
    for arr in (u, ties):
        f = arr.view(np.float32)
        ref = torch.from_numpy(f.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(oracle.f32_to_bf16_bits(f), ref)


def test_invariants_on_workload_rows():
    P.pin_invariants(oracle, _workload_rows())
    P.pin_invariants(oracle, _near_tie_rows())
    big = workloads.WORKLOADS["attn_proj"].linears[0]
    x = workloads.activations(64, big.K, big.x_dist, 0, big.outlier_frac, big.outlier_factor)
    P.pin_invariants(oracle, x[:16])


def test_scale_equivariance():
    rows = workloads.activations(12, 64, "student_t3", 21, 0.05, 50.0)
    P.pin_scale_equivariance(oracle, rows)


def test_closed_forms():
    P.pin_closed_forms(oracle)


def test_permutation_invariance():
    qx, qw = _codes(16, 24, 512, seed=5)
    P.pin_permutation_invariance(oracle, qx, qw)


def test_sanity_bound_against_float_product():
    x = workloads.activations(16, 256, "student_t3", 8, 0.01, 50.0)
    w = workloads.weights(24, 256, 0.02, 9)
    b = workloads.bias(24, 0.01, 10)
    P.pin_sanity_bound(oracle, x, w, b)


def test_codes_never_reach_minus_eight_on_workloads():
    """With denominator 7 the largest quotient rounds to 7, so -8 does not occur."""
    for name in ("tiny",):
        lin = workloads.WORKLOADS[name].linears[0]
        q, _ = oracle.quantize_rows(lin.make_x())
        assert q.min() >= -7 and q.max() <= 7


def test_layer_composition():
    lin = workloads.WORKLOADS["tiny"].linears[0]
    x, w = lin.make_x(), lin.make_w()
    b = workloads.bias(lin.N, 0.01, 2)
    qw, sw = oracle.pack_weight_int4(w)
    y = oracle.w4a4_linear(x, qw, sw, b)
    qx, sx = oracle.quantize_act(x)
    acc = oracle.w4a4_gemm_i32(qx, qw)
    assert np.array_equal(y, oracle.epilogue(acc, sx, sw, b))
    rows = np.array([0, 17, 63])
    assert np.array_equal(oracle.w4a4_linear_rows(x, qw, sw, rows, b), y[rows])


# ---------------------------------------------------------------------------
# hypothesis: random bf16 rows
# ---------------------------------------------------------------------------

_finite_bf16 = st.integers(0, 0xFFFF).filter(lambda b: (b >> 7) & 0xFF != 0xFF)


@settings(max_examples=150, deadline=None)
@given(st.integers(1, 16).flatmap(lambda h: st.lists(_finite_bf16, min_size=2 * h, max_size=2 * h)))
def test_property_random_rows(row):
    rows = np.array([row], dtype=np.uint16)
    P.pin_rational_quantizer(oracle, rows)
    P.pin_invariants(oracle, rows)


# ---------------------------------------------------------------------------
# mutants: plausible mistakes planted in copies of the oracle
# ---------------------------------------------------------------------------


def _ns(**over):
    base = dict(quantize_rows=oracle.quantize_rows, pack_int4=oracle.pack_int4,
                unpack_int4=oracle.unpack_int4, code_gemm=oracle.code_gemm,
                epilogue=oracle.epilogue)
    base.update(over)
    return types.SimpleNamespace(**base)


def _quant_variant(denom=7.0, mode="div", rounding="rne", axis=1, scale_bf16=False):
    def q(x_bits):
        xf = oracle.bf16_bits_to_f32(x_bits)
        a = np.max(np.abs(xf), axis=axis).astype(np.float32)
        s = (a / np.float32(denom)).astype(np.float32)
        if scale_bf16:
            s = oracle.bf16_bits_to_f32(oracle.f32_to_bf16_bits(s))
        if axis == 0:
            s_b = s[None, :]
            s_out = s
        else:
            s_b = s[:, None]
            s_out = s
        with np.errstate(all="ignore"):
            if mode == "div":
                t = (xf / s_b).astype(np.float32)
            else:
                t = (xf * (np.float32(denom) / (a[None, :] if axis == 0 else a[:, None]))).astype(np.float32)
            if rounding == "rne":
                r = np.rint(t)
            elif rounding == "away":
                r = np.sign(t) * np.floor(np.abs(t) + 0.5)
            else:
                r = np.trunc(t)
            r = np.where(np.isfinite(r), r, 0)
        qq = np.clip(r, -8, 7).astype(np.int8)
        qq[np.broadcast_to(s_b == 0, qq.shape)] = 0
        return qq, s_out
    return q


def _pack_swapped(q):
    q = np.asarray(q, dtype=np.int16)
    return ((q[:, 1::2] & 0xF) | ((q[:, 0::2] & 0xF) << 4)).astype(np.uint8)


def _unpack_swapped(p):
    u = oracle.unpack_int4(p)
    out = u.copy()
    out[:, 0::2], out[:, 1::2] = u[:, 1::2], u[:, 0::2]
    return out


def _pack_unsigned_sat(q):
    q = np.clip(np.asarray(q, dtype=np.int16), 0, 15)
    return (q[:, 0::2] | (q[:, 1::2] << 4)).astype(np.uint8)


def _epi(order="pinned", bias=True, bf16_round="rne"):
    def e(acc, sx, sw, bias_bits=None):
        t = np.asarray(acc).astype(np.float32)
        sx = np.asarray(sx, np.float32)
        sw = np.asarray(sw, np.float32)
        if order == "pinned":
            t = (t * sx[:, None]).astype(np.float32) * sw[None, :]
        else:  # combined scale first: a different rounding order
            t = t * (sx[:, None] * sw[None, :]).astype(np.float32)
        t = t.astype(np.float32)
        if bias and bias_bits is not None:
            t = (t + oracle.bf16_bits_to_f32(bias_bits)[None, :]).astype(np.float32)
        if bf16_round == "rne":
            return oracle.f32_to_bf16_bits(t)
        return (t.view(np.uint32) >> 16).astype(np.uint16)
    return e


def _gemm_transposed_w(qx, qw):
    return (qx.astype(np.float64) @ qw.astype(np.float64)).astype(np.int64)


def _gemm_wraps_int16(qx, qw):
    return oracle.code_gemm(qx, qw).astype(np.int16).astype(np.int64)


def _gemm_drops_last_k(qx, qw):
    return oracle.code_gemm(qx[:, :-1], qw[:, :-1])


MUTANTS = {
    "reciprocal_multiply": _ns(quantize_rows=_quant_variant(mode="mul")),
    "denominator_8": _ns(quantize_rows=_quant_variant(denom=8.0)),
    "round_half_away": _ns(quantize_rows=_quant_variant(rounding="away")),
    "truncate": _ns(quantize_rows=_quant_variant(rounding="trunc")),
    "per_column_scale": _ns(quantize_rows=_quant_variant(axis=0)),
    "scale_rounded_to_bf16": _ns(quantize_rows=_quant_variant(scale_bf16=True)),
    "nibbles_swapped": _ns(pack_int4=_pack_swapped, unpack_int4=_unpack_swapped),
    "unsigned_nibbles": _ns(pack_int4=_pack_unsigned_sat),
    "transposed_weight": _ns(code_gemm=_gemm_transposed_w),
    "int16_accumulator": _ns(code_gemm=_gemm_wraps_int16),
    "dropped_k_term": _ns(code_gemm=_gemm_drops_last_k),
    "epilogue_scale_order": _ns(epilogue=_epi(order="combined")),
    "epilogue_drops_bias": _ns(epilogue=_epi(bias=False)),
    "epilogue_truncates_bf16": _ns(epilogue=_epi(bf16_round="trunc")),
}


def _run_pins(impl):
    qx, qw = _codes(4, 6, 64, seed=1)
    qx2, qw2 = _codes(6, 6, 64, seed=2)
    rng = np.random.default_rng(9)
    acc = rng.integers(-300000, 300000, size=(5, 6)).astype(np.int64)
    sx = rng.uniform(0.01, 3, size=5).astype(np.float32)
    sw = rng.uniform(1e-4, 1e-2, size=6).astype(np.float32)
    b = workloads.bias(6, 0.01, 2)
    big_acc = rng.integers(-600000, 600000, size=(5, 6)).astype(np.int64)
    samples = [(m, n) for m in range(5) for n in range(6)]
    checks = [
        lambda: P.pin_golden_quantizer(impl),
        lambda: P.pin_golden_gemm(impl),
        lambda: P.pin_rational_quantizer(impl, _near_tie_rows(8, 16)),
        lambda: P.pin_rational_quantizer(impl, _workload_rows()[:10]),
        lambda: P.pin_brute_force_gemm(impl, qx, qw),
        lambda: P.pin_brute_force_gemm(impl, qx2, qw2),
        lambda: P.pin_extreme_accumulators(impl, 1024),
        lambda: P.pin_epilogue_rational(impl, acc, sx, sw, b, samples),
        lambda: P.pin_epilogue_rational(impl, big_acc, sx, sw, None, samples),
        lambda: P.pin_invariants(impl, _workload_rows()[:10]),
        lambda: P.pin_epilogue_fp64(impl, *_epilogue_stress()),
        lambda: P.pin_closed_forms(impl),
    ]
    failed = []
    for i, c in enumerate(checks):
        try:
            c()
        except (AssertionError, ValueError, IndexError):
            failed.append(i)
    return failed


def test_pins_pass_on_oracle():
    assert _run_pins(_ns()) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    assert _run_pins(MUTANTS[name]), f"no pin caught mutant {name}"
