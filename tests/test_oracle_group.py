"""The group-wise W4A4 part of the CPU oracle against its pins (no GPU needed).

Mutant tests plant plausible mistakes in copies of the oracle, on the CPU, and
check that at least one pin catches each of them.
"""

import types

import numpy as np
import pytest

import oracle
from paper_2609_33601_amd import workloads
from tests import oracle_pins_group as PG


def _rows(n=12, K=256, seed=3):
    x = workloads.activations(n, K, "student_t3", seed, 0.05, 50.0)
    g = workloads.activations(4, K, "gelu_normal", seed + 1, 0.05, 30.0)
    rng = np.random.default_rng(seed)
    # rows whose groups sit on the half-integer decision points: group absmax 7 * 2^e -> s = 2^e
    ties = []
    for _ in range(4):
        v = (rng.integers(-7, 7, size=K) + 0.5) * 2.0 ** -3
        v[::64] = 7 * 2.0 ** -3
        f = v.astype(np.float32)
        ties.append(((f.view(np.uint32) + 0x8000) >> 16).astype(np.uint16))
    z = x[:1].copy()
    z[0, 64:128] = 0  # one all-zero group
    return np.concatenate([x, g, np.stack(ties), z])


def _run_pins(impl):
    PG.pin_golden_group(impl)
    rows = _rows()
    for G in oracle.GROUP_SIZES:
        PG.pin_rational_group_quantizer(impl, rows[:, :2 * G], G)
        PG.pin_group_brute_force(impl, G)
        PG.pin_group_locality(impl, rows, G)
        PG.pin_group_invariants(impl, rows, G)
    PG.pin_rational_group_sum(impl)
    PG.pin_group_epilogue_rational(impl)
    w = workloads.weights(10, 128, 0.02, 5)
    PG.pin_reduces_to_per_token(impl, rows[:, :128], w, workloads.bias(10, 0.01, 6))


def test_pins_pass_on_oracle():
    _run_pins(oracle)


def test_layer_composition():
    x = _rows()
    w = workloads.weights(20, 256, 0.02, 9)
    b = workloads.bias(20, 0.01, 10)
    for G in oracle.GROUP_SIZES:
        qw, sw = oracle.pack_weight_int4_group(w, G)
        y = oracle.w4a4g_linear(x, qw, sw, G, b)
        qx, sx = oracle.quantize_act_group(x, G)
        S = oracle.group_sum(oracle.group_code_gemm(oracle.unpack_int4(qx), oracle.unpack_int4(qw), G), sx, sw)
        assert np.array_equal(y, oracle.group_epilogue(S, b))
        assert np.array_equal(oracle.w4a4g_gemm_f32(qx, sx, qw, sw, G), S)
        rows = np.array([0, 7, len(x) - 1])
        assert np.array_equal(oracle.w4a4g_linear_rows(x, qw, sw, G, rows, b), y[rows])


def test_group_scales_are_finer_than_per_token():
    """A sanity property of the readings: with per-group scales the quantisation error is never larger."""
    x = _rows()
    xf = (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    qt, st = oracle.quantize_rows(x)
    qg, sg = oracle.quantize_rows_group(x, 64)
    et = np.abs(xf - qt * st[:, None].astype(np.float64))
    eg = np.abs(xf - qg * np.repeat(sg.astype(np.float64), 64, axis=1))
    assert eg.sum() <= et.sum()


# ---------------------------------------------------------------------------
# mutants
# ---------------------------------------------------------------------------


def _ns(**over):
    base = {n: getattr(oracle, n) for n in ("quantize_rows_group", "group_code_gemm", "group_sum",
                                            "group_epilogue", "pack_int4", "unpack_int4")}
    base.update(over)
    return types.SimpleNamespace(**base)


def _q_per_token(x_bits, G):
    q, s = oracle.quantize_rows(x_bits)
    return q, np.repeat(s[:, None], x_bits.shape[1] // G, axis=1)


def _q_strided(x_bits, G):
    """Groups taken as k mod (K/G) instead of consecutive k."""
    R, K = x_bits.shape
    ng = K // G
    perm = np.arange(K).reshape(G, ng).T.reshape(-1)
    q, s = oracle.quantize_rows_group(x_bits[:, perm], G)
    out = np.empty_like(q)
    out[:, perm] = q
    return out, s


def _q_mul_7_over_absmax(x_bits, G):
    """x * fl32(7 / absmax) instead of fl32(x / s)."""
    R, K = x_bits.shape
    xf = oracle.bf16_bits_to_f32(x_bits).reshape(R, K // G, G)
    a = np.max(np.abs(xf), axis=2).astype(np.float32)
    s = (a / np.float32(7)).astype(np.float32)
    with np.errstate(divide="ignore"):
        r = np.where(a > 0, (np.float32(7) / a).astype(np.float32), 0).astype(np.float32)
    q = np.clip(np.rint((xf * r[:, :, None]).astype(np.float32)), -8, 7).astype(np.int8)
    return q.reshape(R, K), s


def _sum_reverse(acc, s_x, s_w):
    return oracle.group_sum(acc[:, :, ::-1], s_x[:, ::-1], s_w[:, ::-1])


def _sum_fp64(acc, s_x, s_w):
    t = acc.astype(np.float64) * s_x.astype(np.float64)[:, None, :] * s_w.astype(np.float64)[None, :, :]
    return t.sum(axis=2).astype(np.float32)


def _sum_scale_product(acc, s_x, s_w):
    S = np.zeros(acc.shape[:2], np.float32)
    for g in range(acc.shape[2]):
        sxw = (s_x[:, g][:, None] * s_w[:, g][None, :]).astype(np.float32)
        S = (S + (acc[:, :, g].astype(np.float32) * sxw).astype(np.float32)).astype(np.float32)
    return S


def _sum_first_scale(acc, s_x, s_w):
    ng = acc.shape[2]
    tot = acc.sum(axis=2, keepdims=True)
    return oracle.group_sum(tot, s_x[:, :1], s_w[:, :1]) if ng else None


def _gemm_half_groups(qx, qw, G):
    acc = oracle.group_code_gemm(qx, qw, G // 2)
    return acc[:, :, 0::2] + 0 * acc[:, :, 1::2]


MUTANTS = {
    "per_token_scale": _ns(quantize_rows_group=_q_per_token),
    "strided_groups": _ns(quantize_rows_group=_q_strided),
    "multiply_by_7_over_absmax": _ns(quantize_rows_group=_q_mul_7_over_absmax),
    "groups_summed_in_reverse": _ns(group_sum=_sum_reverse),
    "fp64_group_sum": _ns(group_sum=_sum_fp64),
    "scale_product_first": _ns(group_sum=_sum_scale_product),
    "one_scale_for_all_groups": _ns(group_sum=_sum_first_scale),
    "drops_half_of_each_group": _ns(group_code_gemm=_gemm_half_groups),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    with pytest.raises(AssertionError):
        _run_pins(MUTANTS[name])
