"""GPU parity of group-wise W4A4 on the BF6 engine (G = 64, 128) against the CPU oracle.

Bars: codes (decoded from the BF6 operand) and fp32 group scales bit-exact;
the fp32 group sum S (jq_w4a4g_f6_gemm_f32) bit-exact, since both sides add
the same rounded terms in the same order; bf16 outputs within 1 bf16 ulp of
the oracle (expected bit-identical) and bit-identical to the int8 engine's
group-wise layer.  Full-size layers are checked whole against the int8 engine
and on sampled output rows against the oracle.
"""

import numpy as np
import pytest

import oracle
from paper_2609_33601_amd import jq, workloads
from tests.test_gpu_f6 import decode_f6
from tests.test_gpu_parity import _edge_rows, assert_bf16_close, dev_bf16, say  # noqa: F401

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

GS = (64, 128)


def padded_ref_codes(q_packed, rows, K):
    c = oracle.unpack_int4(q_packed).astype(np.int64)
    out = np.zeros((32 * ((rows + 31) // 32), 128 * ((K + 127) // 128)), np.int64)
    out[:rows, :K] = c
    return out


def rand_group_operands(rows, K, G, seed):
    """Random codes -8..7 and positive random scales [rows, K/G] (some zero)."""
    rng = np.random.default_rng(seed)
    q = rng.integers(0, 256, size=(rows, K // 2), dtype=np.uint8)
    s = rng.uniform(0.5, 2.0, size=(rows, K // G)).astype(np.float32) * np.float32(2.0) ** rng.integers(
        -12, 4, size=(rows, K // G)).astype(np.float32)
    s[rng.random(s.shape) < 0.02] = 0.0
    return q, s.astype(np.float32)


# ---------------------------------------------------------------------------
# group quantiser into the BF6 layout
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("M,K,G", [(1, 64, 64), (33, 128, 128), (64, 576, 64), (100, 3072, 64), (37, 4224, 128),
                                   (8, 12288, 64), (5, 65536, 128)])
def test_group_quantize_f6_matches_oracle(M, K, G):
    bits = workloads.activations(M, K, "student_t3", M + K + G, 0.01, 50.0)
    say("group quantize f6", M, K, G)
    xf6, s = jq.jq_quantize_act_group_f6(dev_bf16(bits), G)
    torch.cuda.synchronize()
    rq, rs = oracle.quantize_act_group(bits, G)
    sb, rsb = s.cpu().numpy().view(np.uint32), rs.view(np.uint32)
    assert np.array_equal(sb, rsb), f"{int((sb != rsb).sum())} scales differ"
    codes = decode_f6(xf6.cpu().numpy(), M, K)
    assert np.array_equal(codes, padded_ref_codes(rq, M, K))


@pytest.mark.parametrize("K,G", [(128, 64), (576, 64), (3072, 128), (12288, 64)])
def test_group_quantize_f6_edge_rows(K, G):
    bits = _edge_rows(K, seed=K + 3 * G)
    say("group quantize f6 edge rows", bits.shape, G)
    xf6, s = jq.jq_quantize_act_group_f6(dev_bf16(bits), G)
    torch.cuda.synchronize()
    rq, rs = oracle.quantize_act_group(bits, G)
    assert np.array_equal(s.cpu().numpy().view(np.uint32), rs.view(np.uint32))
    assert np.array_equal(decode_f6(xf6.cpu().numpy(), bits.shape[0], K), padded_ref_codes(rq, bits.shape[0], K))


# ---------------------------------------------------------------------------
# exact fp32 group sum
# ---------------------------------------------------------------------------


def f6_group_sum(qx, sx, qw, sw, G):
    xf6 = jq.jq_int4_to_f6(torch.from_numpy(qx).cuda())
    wf6 = jq.jq_int4_to_f6_weight(torch.from_numpy(qw).cuda())
    S = jq.jq_w4a4g_f6_gemm_f32(xf6, torch.from_numpy(sx).cuda(), wf6, torch.from_numpy(sw).cuda(), G)
    torch.cuda.synchronize()
    return S.cpu().numpy()


@pytest.mark.parametrize("M,N,K,G", [(1, 1, 64, 64), (3, 5, 128, 128), (32, 32, 192, 64), (129, 255, 320, 64),
                                     (257, 130, 512, 128), (300, 520, 1088, 64), (1000, 700, 2048, 128),
                                     (2100, 1500, 448, 64)])
def test_group_f6_sum_random_operands(M, N, K, G):
    say("group f6 sum", M, N, K, G)
    qx, sx = rand_group_operands(M, K, G, seed=M + K)
    qw, sw = rand_group_operands(N, K, G, seed=N + 2 * K)
    got = f6_group_sum(qx, sx, qw, sw, G)
    ref = oracle.w4a4g_gemm_f32(qx, sx, qw, sw, G)
    bad = np.argwhere(got.view(np.uint32) != ref.view(np.uint32))
    assert bad.size == 0, f"{len(bad)} sums differ, first {bad[:4].tolist()}"


# ---------------------------------------------------------------------------
# whole layer
# ---------------------------------------------------------------------------


def group_layers(x_bits, w_bits, b_bits, G):
    """The group-wise layer on the BF6 engine and on the int8 engine, same inputs."""
    x = dev_bf16(x_bits)
    wq, sw = jq.jq_pack_weight_int4_group(dev_bf16(w_bits), G)
    wf6 = jq.jq_int4_to_f6_weight(wq)
    b = None if b_bits is None else dev_bf16(b_bits)
    y6 = jq.jq_w4a4g_f6_linear(x, wf6, sw, G, b)
    y8 = jq.jq_w4a4g_linear(x, wq, sw, G, b)
    torch.cuda.synchronize()
    return y6, y8, wq.cpu().numpy(), sw.cpu().numpy()


@pytest.mark.parametrize("M,K,N,G,bias", [(77, 3072, 130, 64, True), (1, 64, 1, 64, False), (5, 128, 4096, 128, True),
                                          (300, 1088, 260, 64, False), (513, 256, 777, 128, True),
                                          (257, 4160, 300, 64, True)])
def test_group_f6_linear_ragged(M, K, N, G, bias):
    say("group f6 linear ragged", M, K, N, G, bias)
    x = workloads.activations(M, K, "student_t3", M + 11, 0.01, 50.0)
    w = workloads.weights(N, K, 0.02, N + 13)
    b = workloads.bias(N, 0.01, 17) if bias else None
    y6, y8, wq, sw = group_layers(x, w, b, G)
    assert torch.equal(y6.view(torch.int16), y8.view(torch.int16))
    assert_bf16_close(jq.bf16_bits(y6), oracle.w4a4g_linear(x, wq, sw, G, b), f"group f6 {M}x{K}->{N} G={G}")


def test_group_f6_gemm_matches_linear():
    """GEMM on a separately quantised operand equals the whole linear."""
    lin = workloads.WORKLOADS["dllm_block"].linears[0]
    M, G = 512, 128
    x = dev_bf16(lin.make_x()[:M])
    wq, sw = jq.jq_pack_weight_int4_group(dev_bf16(lin.make_w()[:1024]), G)
    wf6 = jq.jq_int4_to_f6_weight(wq)
    xf6, s = jq.jq_quantize_act_group_f6(x, G)
    y1 = jq.jq_w4a4g_f6_gemm(xf6, s, wf6, sw, G)
    y2 = jq.jq_w4a4g_f6_linear(x, wf6, sw, G)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


@pytest.mark.parametrize("G", GS)
def test_group_f6_linear_edge_rows(G):
    """Edge rows (zero, subnormal, near-max, ties) through the BF6 group-wise layer."""
    say("group f6 linear edge rows", G)
    K, N = 256, 96
    x = _edge_rows(K, seed=5)
    w = workloads.weights(N, K, 0.02, 6)
    b = workloads.bias(N, 0.01, 7)
    y6, y8, wq, sw = group_layers(x, w, b, G)
    assert torch.equal(y6.view(torch.int16), y8.view(torch.int16))
    assert_bf16_close(jq.bf16_bits(y6), oracle.w4a4g_linear(x, wq, sw, G, b), f"group{G} edge rows")
