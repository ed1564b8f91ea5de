"""GPU parity of the W1.58A4 path (ternary weights, int4 activations) against the CPU oracle.

Bars: ternary codes, fp32 weight scales and int32 accumulators bit-exact;
bf16 outputs within 1 bf16 ulp of the oracle (expected bit-identical: the
epilogue follows the same rounding sequence).  Full-size layers are checked
here on whole packed weights; every output and accumulator of the full-size
layers is compared with the oracle in tests/test_gpu_full_oracle.py.
"""

import numpy as np
import pytest

import oracle
from paper_2609_33601_amd import jq, workloads
from tests import oracle_pins as P
from tests.test_gpu_parity import _edge_rows, _gpu, _sample_rows, assert_bf16_close, dev_bf16, fp_bits, say  # noqa: F401

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def gpu_pack_ternary(bits):
    wt, g = jq.jq_pack_weight_ternary(dev_bf16(bits))
    torch.cuda.synchronize()
    return wt.cpu().numpy(), g.cpu().numpy()


def assert_ternary_equal(bits, wt, g, what):
    rt, rg = oracle.pack_weight_ternary(bits)
    assert np.array_equal(g.view(np.uint32), rg.view(np.uint32)), \
        f"{what}: scale bits differ at rows {np.argwhere(g.view(np.uint32) != rg.view(np.uint32))[:4].ravel().tolist()}"
    bad = np.argwhere(wt != rt)
    assert bad.size == 0, f"{what}: {len(bad)} packed bytes differ, first {bad[:4].tolist()}"


def rand_ternary_packed(rows, K, seed):
    t = np.random.default_rng(seed).integers(-1, 2, size=(rows, K)).astype(np.int8)
    return oracle.pack_ternary(t)


def rand_int4_packed(rows, K, seed):
    return np.random.default_rng(seed).integers(0, 256, size=(rows, K // 2), dtype=np.uint8)


# ---------------------------------------------------------------------------
# ternary weight quantiser
# ---------------------------------------------------------------------------


def test_pack_ternary_golden_examples():
    from tests.golden import fixtures

    cases = fixtures.load("ternary_examples.txt")
    names = ("tern1_basic", "tern2_ties", "tern3_zero_row", "tern4_clamp_negative")
    # tiling a row 8 times keeps its mean, so the codes and the scale stay those of the 8-element example
    bits = np.stack([np.tile(P.exact_bf16_bits(cases[n]["w"]), 8) for n in names])
    wt, g = gpu_pack_ternary(bits)
    for i, n in enumerate(names):
        c = cases[n]
        assert wt[i].tolist() == c["packed"] * 8, n
        assert int(g[i:i + 1].view(np.uint32)[0]) == c["g_bits"][0], n
    assert_ternary_equal(bits, wt, g, "golden")


def _ternary_edge_rows(K, seed):
    rng = np.random.default_rng(seed)
    rows = [workloads.weights(1, K, 0.02, seed)[0], np.zeros(K, np.uint16)]
    sub = rng.integers(1, 0x80, size=K).astype(np.uint16)                 # subnormals only
    sub[rng.random(K) < 0.5] |= 0x8000
    rows.append(sub)
    rows.append(rng.integers(0x7F00, 0x7F80, size=K).astype(np.uint16))  # near bf16 max
    one = np.zeros(K, np.uint16)
    one[K // 2] = 0xC040                                                  # single -3
    rows.append(one)
    # exact decision points: the block 6 4.5 1.5 1.5 3 4.5 3 0 has g = 3, 1.5/g = 0.5, 4.5/g = 1.5
    base = np.tile(np.array([6, 4.5, 1.5, 1.5, 3, 4.5, 3, 0], np.float32), K // 8)
    for e in (-9, 0, 7):
        v = base * np.float32(2.0 ** e) * rng.choice([-1.0, 1.0], size=K).astype(np.float32)
        rows.append(fp_bits(v[rng.permutation(K)]))
    rows.append(np.where(rng.random(K) < 0.5, 0x3F40, 0xBF40).astype(np.uint16))  # +-0.75: g = 0.75
    return np.stack(rows)


@pytest.mark.parametrize("K", [64, 192, 576, 3072, 12288, 65536])
def test_pack_ternary_edge_rows(K):
    bits = _ternary_edge_rows(K, seed=K)
    say("pack ternary edge rows", bits.shape)
    wt, g = gpu_pack_ternary(bits)
    assert_ternary_equal(bits, wt, g, f"edge K={K}")


@pytest.mark.parametrize("lin", [l for wl in workloads.WORKLOADS.values() for l in wl.linears],
                         ids=lambda l: f"{l.name}-W{l.N}x{l.K}")
def test_pack_ternary_full_workloads(lin):
    say("pack ternary", lin.name, lin.N, lin.K)
    bits = lin.make_w()
    wt, g = gpu_pack_ternary(bits)
    assert_ternary_equal(bits, wt, g, lin.name + " ternary weight")


# ---------------------------------------------------------------------------
# exact accumulators
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("M,N,K", [(1, 1, 64), (3, 5, 128), (16, 16, 64), (257, 255, 192),
                                   (300, 520, 1024), (256, 256, 3072), (513, 1000, 640),
                                   (1, 4099, 128), (2049, 3, 320), (130, 300, 12288)])
def test_w158a4_gemm_i32_random_codes(M, N, K):
    say("w158a4 gemm i32", M, N, K)
    qx = rand_int4_packed(M, K, seed=M * 7 + K)
    wt = rand_ternary_packed(N, K, seed=N * 11 + K)
    acc = jq.jq_w158a4_gemm_i32(torch.from_numpy(qx).cuda(), torch.from_numpy(wt).cuda())
    torch.cuda.synchronize()
    ref = oracle.w158a4_gemm_i32(qx, wt)
    bad = np.argwhere(acc.cpu().numpy() != ref)
    assert bad.size == 0, f"{len(bad)} accumulators differ, first {bad[:4].tolist()}"


@pytest.mark.parametrize("code_x,code_t", [(-8, -1), (7, -1), (-8, 1)])
def test_w158a4_gemm_i32_extreme_codes_max_k(code_x, code_t):
    K = 65536
    M, N = 300, 260
    qx = np.full((M, K // 2), (code_x & 0xF) | ((code_x & 0xF) << 4), np.uint8)
    f = code_t & 3
    wt = np.full((N, K // 4), f | (f << 2) | (f << 4) | (f << 6), np.uint8)
    acc = jq.jq_w158a4_gemm_i32(torch.from_numpy(qx).cuda(), torch.from_numpy(wt).cuda()).cpu().numpy()
    assert np.all(acc == code_x * code_t * K)


# ---------------------------------------------------------------------------
# whole layer
# ---------------------------------------------------------------------------


def _layer(bits_x, bits_w, bits_b):
    wt, g = jq.jq_pack_weight_ternary(dev_bf16(bits_w))
    b = None if bits_b is None else dev_bf16(bits_b)
    y = jq.jq_w158a4_linear(dev_bf16(bits_x), wt, g, b)
    torch.cuda.synchronize()
    return jq.bf16_bits(y), wt.cpu().numpy(), g.cpu().numpy()


@pytest.mark.parametrize("with_bias", [False, True])
def test_w158a4_linear_tiny_workload_full(with_bias):
    lin = workloads.WORKLOADS["tiny"].linears[0]
    x, w = lin.make_x(), lin.make_w()
    b = workloads.bias(lin.N, 0.01, 2) if with_bias else None
    y, wt, g = _layer(x, w, b)
    assert_ternary_equal(w, wt, g, "tiny weight")
    rt, rg = oracle.pack_weight_ternary(w)
    assert_bf16_close(y, oracle.w158a4_linear(x, rt, rg, b), f"w158a4 tiny bias={with_bias}")


@pytest.mark.parametrize("M,K,N,bias", [(77, 3072, 130, True), (1, 64, 1, False), (5, 192, 4096, True),
                                        (300, 1088, 260, False), (513, 256, 777, True)])
def test_w158a4_linear_ragged(M, K, N, bias):
    say("w158a4 linear ragged", M, K, N, bias)
    x = workloads.activations(M, K, "student_t3", M + 3, 0.01, 50.0)
    w = workloads.weights(N, K, 0.02, N + 5)
    b = workloads.bias(N, 0.01, 7) if bias else None
    y, wt, g = _layer(x, w, b)
    assert_bf16_close(y, oracle.w158a4_linear(x, wt, g, b), f"w158a4 ragged {M}x{K}->{N}")


def test_w158a4_linear_edge_rows_outputs():
    """Zero, subnormal, huge and tie activation rows through the whole ternary layer."""
    K, N = 256, 96
    x = _edge_rows(K, seed=5)
    w = workloads.weights(N, K, 0.02, 6)
    b = workloads.bias(N, 0.01, 7)
    y, wt, g = _layer(x, w, b)
    assert_bf16_close(y, oracle.w158a4_linear(x, wt, g, b), "w158a4 edge rows")
