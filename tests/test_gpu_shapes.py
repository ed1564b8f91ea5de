"""Seeded random shapes through both engines, every output against the oracle.

Twenty-four shapes drawn from one fixed seed (sixteen with M and N up to
1500 and K up to 2048; four with M near a multiple of 256 up to 6144, N up
to 12288 and K up to 512; four with K from 6208 to 8192; bias on or off,
heavy-tailed activations with outlier columns) cover the tile and edge
combinations the fixed cases do not name: both tile heights of the int8
GEMM, the BF6 GEMM's block shapes and tile heights, K tails
(K % 128 == 64), and ragged M and N edges.  Each
shape runs through jq_w4a4_linear and jq_w4a4_f6_linear (the weight packed
once and re-encoded for the BF6 engine); both must equal the oracle's bf16
outputs bit for bit, the quantised activations in the int8 workspace must
equal the oracle's codes and scales, and the shape's GEMM plans are logged.
Twelve more shapes each do the same for W1.58A4 and for group-wise W4A4
(G = 64 and 128 alternating, the group sums from the oracle's compiled
form).
"""

import sys

import numpy as np
import pytest

import oracle
from paper_2609_33601_amd import jq, workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def say(*a):
    print("[gpu-shapes]", *a, flush=True)
    sys.stdout.flush()


def _shapes(seed=20260):
    """16 small shapes, 4 with many tiles and short K, 4 with K past 6144."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(24):
        if i < 16:
            M, N, K = int(rng.integers(1, 1501)), int(rng.integers(1, 1501)), 64 * int(rng.integers(1, 33))
        elif i < 20:
            M = 256 * int(rng.integers(12, 25)) - int(rng.integers(0, 40))
            N, K = int(rng.integers(4000, 12289)), 64 * int(rng.integers(2, 9))
        else:
            M, N, K = int(rng.integers(1, 700)), int(rng.integers(1, 700)), 64 * int(rng.integers(97, 129))
        out.append((M, N, K, bool(i % 2), 1000 + i))
    return out


SHAPES = _shapes()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the parity tests need an MI355X")
    yield
    torch.cuda.synchronize()


def test_shapes_cover_tile_variety():
    """The draw includes K tails, both int8 tile heights and both BF6 block shapes."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    heights = {jq.jq_gemm_plan(M, N, K, cus) for M, N, K, _, _ in SHAPES}
    f6 = {jq.jq_f6_gemm_plan(M, N, K, cus) for M, N, K, _, _ in SHAPES}
    assert any(K % 128 == 64 for _, _, K, _, _ in SHAPES)
    assert heights == {112, 128}, heights
    assert {w for w, _ in f6} == {4, 8}, f6
    say("int8 tile heights drawn:", sorted(heights))


@pytest.mark.parametrize("M,N,K,bias,seed", SHAPES, ids=lambda v: str(v))
def test_random_shape_both_engines(M, N, K, bias, seed):
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    say(f"{M}x{K}->{N} bias={bias}: int8 tile rows {jq.jq_gemm_plan(M, N, K, cus)}, "
        f"bf6 (waves, tile rows) {jq.jq_f6_gemm_plan(M, N, K, cus)}")
    x_bits = workloads.activations(M, K, "student_t3", seed, 0.01, 50.0)
    w_bits = workloads.weights(N, K, 0.02, seed + 1)
    b_bits = workloads.bias(N, 0.01, seed + 2) if bias else None
    rwq, rsw = oracle.pack_weight_int4(w_bits)
    rqx, rsx = oracle.quantize_act(x_bits)
    ref = oracle.w4a4_gemm(rqx, rsx, rwq, rsw, b_bits)

    x = jq.bf16_tensor(x_bits, "cuda")
    b = None if b_bits is None else jq.bf16_tensor(b_bits, "cuda")
    wq, sw = jq.jq_pack_weight_int4(jq.bf16_tensor(w_bits, "cuda"))
    ws = torch.empty(jq.jq_w4a4_workspace_bytes(M, K), dtype=torch.uint8, device="cuda")
    y4 = jq.jq_w4a4_linear(x, wq, sw, b, workspace=ws)
    y6 = jq.jq_w4a4_f6_linear(x, jq.jq_int4_to_f6_weight(wq), sw, b)
    torch.cuda.synchronize()
    assert np.array_equal(wq.cpu().numpy(), rwq), "weight codes differ"
    assert np.array_equal(sw.cpu().numpy().view(np.uint32), rsw.view(np.uint32)), "weight scales differ"
    codes = M * K // 2
    off = (codes + 255) // 256 * 256
    assert np.array_equal(ws[:codes].cpu().numpy().reshape(M, K // 2), rqx), "activation codes differ"
    assert np.array_equal(ws[off: off + 4 * M].view(torch.float32).cpu().numpy().view(np.uint32),
                          rsx.view(np.uint32)), "activation scales differ"
    d4 = int(np.count_nonzero(jq.bf16_bits(y4) != ref))
    d6 = int(np.count_nonzero(jq.bf16_bits(y6) != ref))
    assert d4 == 0 and d6 == 0, f"{M}x{K}->{N}: {d4} (int8) and {d6} (bf6) of {M * N} outputs differ"


# ---------------------------------------------------------------------------
# W1.58A4 and group-wise W4A4 on the same kind of draw
# ---------------------------------------------------------------------------


def _small_shapes(n, seed, kmul):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        M, N = int(rng.integers(1, 1501)), int(rng.integers(1, 1501))
        K = kmul * int(rng.integers(1, 4096 // kmul + 1))
        out.append((M, N, K, bool(i % 2), 2000 + i))
    return out


TERNARY_SHAPES = _small_shapes(12, 20261, 64)
# G = 64 takes any K % 64 == 0 (K % 128 == 64 included), G = 128 K rounded up to 128
GROUP_SHAPES = [(M, N, K if G == 64 else -(-K // 128) * 128, bias, seed, G)
                for (M, N, K, bias, seed), G in zip(_small_shapes(12, 20262, 64), [64, 128] * 6)]


@pytest.mark.parametrize("M,N,K,bias,seed", TERNARY_SHAPES, ids=lambda v: str(v))
def test_random_shape_ternary_both_engines(M, N, K, bias, seed):
    say(f"W1.58A4 {M}x{K}->{N} bias={bias}")
    x_bits = workloads.activations(M, K, "student_t3", seed, 0.01, 50.0)
    w_bits = workloads.weights(N, K, 0.02, seed + 1)
    b_bits = workloads.bias(N, 0.01, seed + 2) if bias else None
    rwt, rg = oracle.pack_weight_ternary(w_bits)
    ref = oracle.w158a4_linear(x_bits, rwt, rg, b_bits)

    x = jq.bf16_tensor(x_bits, "cuda")
    b = None if b_bits is None else jq.bf16_tensor(b_bits, "cuda")
    wt, g = jq.jq_pack_weight_ternary(jq.bf16_tensor(w_bits, "cuda"))
    y4 = jq.jq_w158a4_linear(x, wt, g, b)
    y6 = jq.jq_w4a4_f6_linear(x, jq.jq_ternary_to_f6_weight(wt), g, b)
    torch.cuda.synchronize()
    assert np.array_equal(wt.cpu().numpy(), rwt), "ternary codes differ"
    assert np.array_equal(g.cpu().numpy().view(np.uint32), rg.view(np.uint32)), "ternary scales differ"
    d4 = int(np.count_nonzero(jq.bf16_bits(y4) != ref))
    d6 = int(np.count_nonzero(jq.bf16_bits(y6) != ref))
    assert d4 == 0 and d6 == 0, f"{M}x{K}->{N}: {d4} (int8) and {d6} (bf6) of {M * N} outputs differ"


@pytest.mark.parametrize("M,N,K,bias,seed,G", GROUP_SHAPES, ids=lambda v: str(v))
def test_random_shape_group_both_engines(M, N, K, bias, seed, G):
    from oracle import group_sum_c

    say(f"group{G} {M}x{K}->{N} bias={bias}")
    x_bits = workloads.activations(M, K, "student_t3", seed, 0.01, 50.0)
    w_bits = workloads.weights(N, K, 0.02, seed + 1)
    b_bits = workloads.bias(N, 0.01, seed + 2) if bias else None
    rwq, rsw = oracle.pack_weight_int4_group(w_bits, G)
    rqx, rsx = oracle.quantize_act_group(x_bits, G)
    ref = oracle.group_epilogue(group_sum_c.w4a4g_gemm_f32(rqx, rsx, rwq, rsw, G), b_bits)

    x = jq.bf16_tensor(x_bits, "cuda")
    b = None if b_bits is None else jq.bf16_tensor(b_bits, "cuda")
    wq, sw = jq.jq_pack_weight_int4_group(jq.bf16_tensor(w_bits, "cuda"), G)
    y4 = jq.jq_w4a4g_linear(x, wq, sw, G, b)
    y6 = jq.jq_w4a4g_f6_linear(x, jq.jq_int4_to_f6_weight(wq), sw, G, b)
    torch.cuda.synchronize()
    assert np.array_equal(wq.cpu().numpy(), rwq), "weight codes differ"
    assert np.array_equal(sw.cpu().numpy().view(np.uint32), rsw.view(np.uint32)), "weight group scales differ"
    d4 = int(np.count_nonzero(jq.bf16_bits(y4) != ref))
    d6 = int(np.count_nonzero(jq.bf16_bits(y6) != ref))
    assert d4 == 0 and d6 == 0, f"{M}x{K}->{N} G={G}: {d4} (int8) and {d6} (bf6) of {M * N} outputs differ"
