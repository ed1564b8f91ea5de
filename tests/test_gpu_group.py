"""GPU parity of the group-wise W4A4 path (G = 64, 128) against the CPU oracle.

Bars: packed codes and fp32 group scales bit-exact; the fp32 group sum S
(exposed by jq_w4a4g_gemm_f32) bit-exact, since both sides add the same
rounded terms in the same order; bf16 outputs within 1 bf16 ulp (expected
bit-identical).  Full-size layers are checked on whole quantised tensors and on
sampled output rows: the oracle's group product keeps every group's exact
partial sum ([M, N, K/G] integers), which at full size would take tens of GB
and minutes per layer, so only rows are drawn from it there.
"""

import numpy as np
import pytest

import oracle
from paper_2609_33601_amd import jq, workloads
from tests import oracle_pins_group as PG
from tests.test_gpu_parity import _edge_rows, _gpu, assert_bf16_close, dev_bf16, say  # noqa: F401

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

GS = (64, 128)


def gpu_quantize_group(bits, G, weight=False):
    fn = jq.jq_pack_weight_int4_group if weight else jq.jq_quantize_act_group
    q, s = fn(dev_bf16(bits), G)
    torch.cuda.synchronize()
    return q.cpu().numpy(), s.cpu().numpy()


def assert_group_quant_equal(bits, G, q, s, what):
    rq, rs = oracle.quantize_act_group(bits, G)
    bad_s = np.argwhere(s.view(np.uint32) != rs.view(np.uint32))
    assert bad_s.size == 0, f"{what}: {len(bad_s)} scales differ, first {bad_s[:4].tolist()}"
    bad = np.argwhere(q != rq)
    assert bad.size == 0, f"{what}: {len(bad)} packed bytes differ, first {bad[:4].tolist()}"


# ---------------------------------------------------------------------------
# group quantiser
# ---------------------------------------------------------------------------


def test_group_quantize_golden_example():
    from tests.golden import fixtures

    c = fixtures.load("group_examples.txt")["grp_gemm_mini"]
    x = PG._sparse(c["K"][0], c["x_idx"], c["x_val"])[None, :]
    q, s = gpu_quantize_group(x, c["G"][0])
    assert [int(v) for v in s[0].view(np.uint32)] == c["sx_bits"]
    assert_group_quant_equal(x, c["G"][0], q, s, "golden")


@pytest.mark.parametrize("K,G", [(K, G) for K in (128, 576, 3072, 12288, 65536) for G in GS if K % G == 0])
def test_group_quantize_edge_rows(K, G):
    bits = _edge_rows(K, seed=K + G)
    say("group quantize edge rows", bits.shape, G)
    q, s = gpu_quantize_group(bits, G)
    assert_group_quant_equal(bits, G, q, s, f"edge K={K} G={G}")
    qw, sw = gpu_quantize_group(bits, G, weight=True)
    assert np.array_equal(qw, q) and np.array_equal(sw.view(np.uint32), s.view(np.uint32))


@pytest.mark.parametrize("G", GS)
@pytest.mark.parametrize("M,K", [(1, 128), (3, 256), (7, 3072), (13, 12288), (4097, 128)])
def test_group_quantize_ragged_row_counts(M, K, G):
    bits = workloads.activations(M, K, "student_t3", M + K + G, 0.005, 50.0)
    q, s = gpu_quantize_group(bits, G)
    assert_group_quant_equal(bits, G, q, s, f"ragged {M}x{K} G={G}")


def _flux_dit():
    return [(workloads.WORKLOADS[n].linears[0], 64) for n in ("mlp_up", "mlp_down")] + \
           [(workloads.WORKLOADS[n].linears[0], 128) for n in ("attn_proj", "qkv")] + \
           [(l, 128) for l in workloads.WORKLOADS["dllm_block"].linears]


@pytest.mark.parametrize("lin,G", _flux_dit(), ids=lambda v: getattr(v, "name", str(v)))
def test_group_quantize_full_workloads(lin, G):
    say("group quantize full", lin.name, G)
    x = lin.make_x()
    q, s = gpu_quantize_group(x, G)
    assert_group_quant_equal(x, G, q, s, lin.name + " activations")
    w = lin.make_w()
    qw, sw = gpu_quantize_group(w, G, weight=True)
    assert_group_quant_equal(w, G, qw, sw, lin.name + " weight")


# ---------------------------------------------------------------------------
# exact fp32 group sums
# ---------------------------------------------------------------------------


def _rand_operands(M, N, K, G, seed):
    rng = np.random.default_rng(seed)
    qx = rng.integers(0, 256, size=(M, K // 2), dtype=np.uint8)
    qw = rng.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    sx = (rng.uniform(0.5, 2, size=(M, K // G)) * 2.0 ** rng.integers(-12, 4, size=(M, K // G))).astype(np.float32)
    sw = (rng.uniform(0.5, 2, size=(N, K // G)) * 2.0 ** rng.integers(-12, 4, size=(N, K // G))).astype(np.float32)
    return qx, sx, qw, sw


@pytest.mark.parametrize("M,N,K,G", [(M, N, K, G) for (M, N, K) in (
    (1, 1, 128), (3, 5, 256), (16, 16, 128), (257, 255, 384), (300, 520, 1024), (256, 256, 3072),
    (513, 1000, 640), (1, 4099, 128), (2049, 3, 1152), (130, 300, 12288)) for G in GS if K % G == 0])
def test_group_gemm_f32_random_codes(M, N, K, G):
    say("group gemm f32", M, N, K, G)
    qx, sx, qw, sw = _rand_operands(M, N, K, G, seed=M * 7 + N + K + G)
    S = jq.jq_w4a4g_gemm_f32(torch.from_numpy(qx).cuda(), torch.from_numpy(sx).cuda(),
                             torch.from_numpy(qw).cuda(), torch.from_numpy(sw).cuda(), G)
    torch.cuda.synchronize()
    ref = oracle.w4a4g_gemm_f32(qx, sx, qw, sw, G)
    got = S.cpu().numpy()
    bad = np.argwhere(got.view(np.uint32) != ref.view(np.uint32))
    assert bad.size == 0, f"{len(bad)} fp32 sums differ, first {bad[:4].tolist()}"


def test_group_gemm_f32_tail_stage():
    """K % 128 == 64 (possible with G = 64 only): the last stage holds a single group."""
    G = 64
    for K in (64, 192, 1088, 12352):
        qx, sx, qw, sw = _rand_operands(70, 90, K, G, seed=K)
        S = jq.jq_w4a4g_gemm_f32(torch.from_numpy(qx).cuda(), torch.from_numpy(sx).cuda(),
                                 torch.from_numpy(qw).cuda(), torch.from_numpy(sw).cuda(), G).cpu().numpy()
        ref = oracle.w4a4g_gemm_f32(qx, sx, qw, sw, G)
        assert np.array_equal(S.view(np.uint32), ref.view(np.uint32)), K


# ---------------------------------------------------------------------------
# whole layer
# ---------------------------------------------------------------------------


def _layer(bits_x, bits_w, bits_b, G):
    wq, sw = jq.jq_pack_weight_int4_group(dev_bf16(bits_w), G)
    b = None if bits_b is None else dev_bf16(bits_b)
    y = jq.jq_w4a4g_linear(dev_bf16(bits_x), wq, sw, G, b)
    torch.cuda.synchronize()
    return jq.bf16_bits(y), wq.cpu().numpy(), sw.cpu().numpy()


def test_group_linear_golden():
    from tests.golden import fixtures

    G = 64
    c = fixtures.load("group_examples.txt")["grp_gemm_mini"]
    K = c["K"][0]
    x = PG._sparse(K, c["x_idx"], c["x_val"])[None, :]
    w0 = PG.exact_bf16_bits(np.repeat(np.array(c["w0_group_vals"], dtype=np.float64), G))
    w1 = PG._sparse(K, c["w1_idx"], c["w1_val"])
    w = np.stack([w0, w1])
    y, _, _ = _layer(x, w, PG.exact_bf16_bits(c["bias"]), G)
    assert [int(v) for v in y[0]] == c["y_bias_bits"]
    y, _, _ = _layer(x, w, None, G)
    assert [int(v) for v in y[0]] == c["y_bits"]


@pytest.mark.parametrize("M,K,N,bias,G", [c + (G,) for c in (
    (64, 256, 256, True), (77, 3072, 130, True), (1, 128, 1, False), (5, 384, 4096, True),
    (300, 1152, 260, False), (513, 256, 777, True), (40, 1088, 300, True)) for G in GS if c[1] % G == 0])
def test_group_linear_ragged(M, K, N, bias, G):
    say("group linear ragged", M, K, N, bias, G)
    x = workloads.activations(M, K, "student_t3", M + 3, 0.01, 50.0)
    w = workloads.weights(N, K, 0.02, N + 5)
    b = workloads.bias(N, 0.01, 7) if bias else None
    y, wq, sw = _layer(x, w, b, G)
    assert_bf16_close(y, oracle.w4a4g_linear(x, wq, sw, G, b), f"group{G} ragged {M}x{K}->{N}")


@pytest.mark.parametrize("G", GS)
def test_group_linear_edge_rows(G):
    K, N = 256, 96
    x = _edge_rows(K, seed=5)
    w = workloads.weights(N, K, 0.02, 6)
    b = workloads.bias(N, 0.01, 7)
    y, wq, sw = _layer(x, w, b, G)
    assert_bf16_close(y, oracle.w4a4g_linear(x, wq, sw, G, b), f"group{G} edge rows")
