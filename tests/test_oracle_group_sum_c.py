"""The compiled group-wise sums (oracle/group_sum.c) against their pins (no GPU needed).

The GPU tests use the compiled form in place of the numpy oracle's group sums
at full size, so it is pinned here on its own: the hand-worked golden example,
exact rational arithmetic with one fp32 rounding per operation and Python
integers for the accumulators, a closed form on extreme codes, overflow, and
bit-for-bit agreement with the numpy oracle on random operands of several
shapes and partitions.  Copies of the C source with a planted mistake are
compiled on the CPU and must each fail a pin.
"""

import os
import subprocess

import numpy as np
import pytest

import oracle
from oracle import group_sum_c
from tests.golden import fixtures
from tests.oracle_pins import f32_bits
from tests.oracle_pins_group import rational_group_sum


@pytest.fixture(scope="module", autouse=True)
def _built():
    if not os.path.exists(group_sum_c.LIB_PATH):
        group_sum_c.build()


def _operands(M, N, K, G, seed):
    """Random codes -8..7 and scales over a wide exponent range (some zero)."""
    rng = np.random.default_rng(seed)
    qx = rng.integers(-8, 8, size=(M, K)).astype(np.int8)
    qw = rng.integers(-8, 8, size=(N, K)).astype(np.int8)

    def scales(r):
        s = (rng.uniform(0.5, 2.0, size=(r, K // G)) * 2.0 ** rng.integers(-40, 20, size=(r, K // G)))
        s = s.astype(np.float32)
        s[rng.random(s.shape) < 0.03] = 0.0
        return s

    return qx, scales(M), qw, scales(N)


def _numpy_oracle(qx, sx, qw, sw, G):
    return oracle.group_sum(oracle.group_code_gemm(qx, qw, G), sx, sw)


def _same_bits(a, b):
    return np.array_equal(np.asarray(a, np.float32).view(np.uint32), np.asarray(b, np.float32).view(np.uint32))


# ---------------------------------------------------------------------------
# pins, each taking the rectangle function of one build
# ---------------------------------------------------------------------------


def pin_golden(fn):
    c = fixtures.load("group_examples.txt")["grp_gemm_mini"]
    K, G = c["K"][0], c["G"][0]
    qx = np.zeros((1, K), np.int8)
    qx[0, c["qx_idx"]] = c["qx_val"]
    qw = np.zeros((2, K), np.int8)
    qw[0, :] = 7
    qw[1, c["w1_idx"]] = [-7, 7, 7, 7, -7]  # the fixture's w1 codes
    bits = lambda key: np.array(c[key], np.uint32).view(np.float32)
    sx = bits("sx_bits")[None, :]
    sw = np.stack([bits("sw0_bits"), bits("sw1_bits")])
    S = group_sum_c.group_sum_codes(qx, sx, qw, sw, G, fn=fn)
    assert [f32_bits(float(v)) for v in S[0]] == c["S_bits"], S


def pin_rational(fn, M=9, N=23, G=16, ng=7, seed=11):
    qx, sx, qw, sw = _operands(M, N, ng * G, G, seed)
    S = group_sum_c.group_sum_codes(qx, sx, qw, sw, G, tile=(4, 8), fn=fn)
    for m in range(M):
        for n in range(N):
            acc = [sum(int(qx[m, k]) * int(qw[n, k]) for k in range(g * G, (g + 1) * G)) for g in range(ng)]
            ref = rational_group_sum(acc, sx[m], sw[n])
            assert float(S[m, n]) == float(ref), (m, n, float(S[m, n]), float(ref))


def pin_extreme_codes(fn):
    """-8 times -8 everywhere: every group's accumulator is 64 G; with unit
    scales the sum over ng groups is 64 G ng exactly (below 2^24)."""
    G, ng = 128, 96
    qx = np.full((3, G * ng), -8, np.int8)
    qw = np.full((5, G * ng), -8, np.int8)
    S = group_sum_c.group_sum_codes(qx, np.ones((3, ng), np.float32), qw, np.ones((5, ng), np.float32), G, fn=fn)
    assert np.all(S == np.float32(64 * G * ng)), S
    # a scale near the fp32 maximum overflows the first product to +inf
    sx = np.ones((3, ng), np.float32)
    sx[1, 5] = np.float32(3.0e38)
    S = group_sum_c.group_sum_codes(qx, sx, qw, np.ones((5, ng), np.float32), G, fn=fn)
    assert np.all(np.isposinf(S[1])) and np.all(S[[0, 2]] == np.float32(64 * G * ng))


def pin_numpy_oracle(fn):
    for (M, N, K, G, tile, seed) in [(37, 130, 256, 64, (32, 64), 1), (5, 3, 384, 128, (32, 64), 2),
                                     (64, 65, 1152, 64, (7, 5), 3), (3, 200, 4096, 128, (1, 64), 4),
                                     (17, 9, 96, 32, (100, 100), 5)]:
        qx, sx, qw, sw = _operands(M, N, K, G, seed)
        S = group_sum_c.group_sum_codes(qx, sx, qw, sw, G, tile=tile, fn=fn)
        assert _same_bits(S, _numpy_oracle(qx, sx, qw, sw, G)), (M, N, K, G)


def _run_pins(fn):
    pin_golden(fn)
    pin_rational(fn)
    pin_extreme_codes(fn)
    pin_numpy_oracle(fn)


def test_pins_pass_on_compiled_oracle():
    _run_pins(group_sum_c.lib())


def test_partition_does_not_change_any_output():
    qx, sx, qw, sw = _operands(45, 77, 640, 64, 7)
    ref = group_sum_c.group_sum_codes(qx, sx, qw, sw, 64, tile=(45, 77), threads=1)
    for tile in [(1, 1), (3, 8), (32, 64), (64, 7)]:
        for threads in (1, 4):
            assert _same_bits(group_sum_c.group_sum_codes(qx, sx, qw, sw, 64, tile=tile, threads=threads), ref)


def test_empty_sides():
    qx, sx, qw, sw = _operands(4, 6, 128, 64, 8)
    assert group_sum_c.group_sum_codes(qx[:0], sx[:0], qw, sw, 64).shape == (0, 6)
    assert group_sum_c.group_sum_codes(qx, sx, qw[:0], sw[:0], 64).shape == (4, 0)


def test_packed_entry_matches_numpy_oracle_on_quantised_layer():
    """From bf16 tensors through the oracle's group quantiser, packed codes in."""
    from paper_2609_33601_amd import workloads

    x = workloads.activations(70, 1024, "student_t3", 3, 0.01, 50.0)
    w = workloads.weights(90, 1024, 0.02, 4)
    for G in oracle.GROUP_SIZES:
        qx, sx = oracle.quantize_act_group(x, G)
        qw, sw = oracle.pack_weight_int4_group(w, G)
        assert _same_bits(group_sum_c.w4a4g_gemm_f32(qx, sx, qw, sw, G), oracle.w4a4g_gemm_f32(qx, sx, qw, sw, G))


# ---------------------------------------------------------------------------
# mutants of the C source
# ---------------------------------------------------------------------------

MUTANTS = {
    "scale_product_first": ("t = t * sx[m * ng + g];\n                t = t * sw[n * ng + g];",
                            "t = t * (sx[m * ng + g] * sw[n * ng + g]);"),
    "fp64_running_sum": ("float s = 0.0f;", "double s = 0.0;"),
    "groups_in_reverse": ("for (int64_t g = 0; g < ng; ++g)", "for (int64_t g = ng - 1; g >= 0; --g)"),
    "one_activation_scale_per_row": ("t = t * sx[m * ng + g];", "t = t * sx[m * ng];"),
    "drops_last_code_of_each_group": ("for (int64_t k = 0; k < G; ++k)", "for (int64_t k = 0; k + 1 < G; ++k)"),
    "fp64_partial": ("float t = (float)acc;\n                t = t * sx[m * ng + g];\n"
                     "                t = t * sw[n * ng + g];",
                     "float t = (float)((double)acc * sx[m * ng + g] * sw[n * ng + g]);"),
    "weight_codes_reversed_in_group": ("acc += (int32_t)a[k] * (int32_t)b[k];",
                                       "acc += (int32_t)a[k] * (int32_t)b[G - 1 - k];"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(group_sum_c.SOURCE).read()
    assert src.count(old) == 1, name
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / "mutant.so"
    subprocess.run(["gcc", *group_sum_c.CFLAGS, str(path), "-o", str(so)], check=True)
    with pytest.raises(AssertionError):
        _run_pins(group_sum_c.load(str(so)))
