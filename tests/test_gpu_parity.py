"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bars: packed int4 codes, fp32 scales and int32 accumulators bit-exact; bf16
outputs within 1 bf16 ulp of the oracle (and in fact expected bit-identical,
since the kernel follows the same rounding sequence).  Full-size workloads are
checked here on whole quantised tensors; every output and accumulator of the
full-size layers is compared with the oracle in tests/test_gpu_full_oracle.py.
"""

import os
import sys

import numpy as np
import pytest

import oracle
from paper_2609_33601_amd import jq, workloads
from tests import oracle_pins as P

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def say(*a):
    print("[gpu-parity]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the parity tests need an MI355X")
    if not os.path.exists(jq.LIB_PATH):
        pytest.fail("libjq.so is not built")
    name = torch.cuda.get_device_properties(0).gcnArchName
    say("device", torch.cuda.get_device_name(0), name)
    yield
    torch.cuda.synchronize()


# ---------------------------------------------------------------------------
# helpers
# ---------------------------------------------------------------------------


def dev_bf16(bits):
    return jq.bf16_tensor(bits, "cuda")


def gpu_quantize(bits, weight=False):
    x = dev_bf16(bits)
    fn = jq.jq_pack_weight_int4 if weight else jq.jq_quantize_act
    q, s = fn(x)
    torch.cuda.synchronize()
    return q.cpu().numpy(), s.cpu().numpy()


def assert_quant_equal(bits, q, s, what):
    rq, rs = oracle.quantize_act(bits)
    assert np.array_equal(s.view(np.uint32), rs.view(np.uint32)), f"{what}: scale bits differ"
    bad = np.argwhere(q != rq)
    assert bad.size == 0, f"{what}: {len(bad)} packed bytes differ, first {bad[:4].tolist()}"


def ulp_bf16(v):
    a = np.abs(v)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    ulp = np.exp2(e - 7)
    return np.where(a >= 2.0 ** -126, ulp, 2.0 ** -133)


def assert_bf16_close(y_bits, ref_bits, what):
    y = oracle.bf16_bits_to_f32(y_bits).astype(np.float64)
    r = oracle.bf16_bits_to_f32(ref_bits).astype(np.float64)
    fin = np.isfinite(r)
    # non-finite references (overflow to inf on huge rows) must match bit for bit
    assert np.array_equal(y_bits[~fin], ref_bits[~fin]), f"{what}: non-finite outputs differ"
    assert np.all(np.isfinite(y[fin])), f"{what}: GPU produced non-finite outputs"
    err = np.where(fin, np.abs(np.where(fin, y, 0) - np.where(fin, r, 0)), 0)
    bad = np.argwhere(err > ulp_bf16(np.where(fin, r, 1.0)))
    assert bad.size == 0, f"{what}: {len(bad)} outputs beyond 1 bf16 ulp, first {bad[:4].tolist()}"
    exact = np.mean(y_bits == ref_bits)
    say(f"{what}: bit-identical fraction {exact:.6f}")


def rand_packed(rows, K, seed):
    return np.random.default_rng(seed).integers(0, 256, size=(rows, K // 2), dtype=np.uint8)


def fp_bits(vals):
    """bf16 bit patterns of float values (they must be bf16-representable)."""
    f = np.asarray(vals, dtype=np.float32)
    u = f.view(np.uint32)
    assert np.all(u & 0xFFFF == 0)
    return (u >> 16).astype(np.uint16)


# ---------------------------------------------------------------------------
# quantiser
# ---------------------------------------------------------------------------


def test_quantize_golden_examples():
    from tests.golden import fixtures

    cases = fixtures.load("quantizer_examples.txt")
    rows = []
    for name in ("ex1_ties", "ex2_division_not_reciprocal", "ex3_zero_row", "ex4_negative_max"):
        rows.append(np.concatenate([P.exact_bf16_bits(cases[name]["x"]), np.zeros(56, np.uint16)]))
    bits = np.stack(rows)
    q, s = gpu_quantize(bits)
    for i, name in enumerate(("ex1_ties", "ex2_division_not_reciprocal", "ex3_zero_row", "ex4_negative_max")):
        c = cases[name]
        assert q[i, :4].tolist() == c["packed"], name
        assert np.all(q[i, 4:] == 0), name
        assert int(s[i:i + 1].view(np.uint32)[0]) == c["s_bits"][0], name
    assert_quant_equal(bits, q, s, "golden")


def _edge_rows(K, seed):
    rng = np.random.default_rng(seed)
    rows = []
    rows.append(workloads.activations(1, K, "normal", seed)[0])
    rows.append(np.zeros(K, np.uint16))                                   # zero row
    sub = rng.integers(1, 0x80, size=K).astype(np.uint16)                 # subnormals only
    sub[rng.random(K) < 0.5] |= 0x8000
    rows.append(sub)
    tiny = sub.copy()
    tiny[:] = 0x0001
    tiny[K // 3] = 0x8001                                                 # smallest subnormal row
    rows.append(tiny)
    big = rng.integers(0x7F00, 0x7F80, size=K).astype(np.uint16)          # near bf16 max
    rows.append(big)
    rows.append(np.where(rng.random(K) < 0.5, 0x3F40, 0xBF40).astype(np.uint16))  # +-0.75
    # exact ties: absmax 7 * 2^e gives s = 2^e, then x = (k + 1/2) 2^e
    e = -3
    ks = rng.integers(-7, 7, size=K) + 0.5
    v = (ks * 2.0 ** e).astype(np.float32)
    v[0] = 7 * 2.0 ** e
    rows.append(fp_bits(v))
    # reciprocal-sensitive rows: absmax 1, many 0.5 / 0.25 / 1.5 * 2^-k
    v = rng.choice([0.5, -0.5, 0.25, 1.5 * 0.125, -0.0625, 0.125, 0.0], size=K).astype(np.float32)
    v[K // 2] = 1.0
    rows.append(fp_bits(v))
    # near-tie rows around (k + 1/2) * absmax / 7 for random absmax
    for t in range(4):
        a = np.float32(rng.uniform(0.1, 100))
        vals = ((rng.integers(-7, 7, size=K) + 0.5) * (np.float64(a) / 7)).astype(np.float32)
        b = ((vals.view(np.uint32) + 0x8000) >> 16).astype(np.int64) + rng.integers(-1, 2, size=K)
        b[t] = int(np.float32(a).view(np.uint32)) >> 16
        rows.append(b.astype(np.uint16))
    one = np.zeros(K, np.uint16)
    one[-1] = 0xC0E0                                                       # single -7 at the end
    rows.append(one)
    rows.append(workloads.activations(1, K, "student_t3", seed + 1, 0.01, 50.0)[0])
    return np.stack(rows)


@pytest.mark.parametrize("K", [64, 256, 576, 1024, 3072, 4160, 12288, 16384, 20480])
def test_quantize_edge_rows(K):
    bits = _edge_rows(K, seed=K)
    say("quantize edge rows", bits.shape)
    q, s = gpu_quantize(bits)
    assert_quant_equal(bits, q, s, f"edge K={K}")
    qw, sw = gpu_quantize(bits, weight=True)
    assert np.array_equal(qw, q) and np.array_equal(sw.view(np.uint32), s.view(np.uint32))


@pytest.mark.parametrize("M,K", [(1, 64), (3, 128), (7, 3072), (13, 12288), (4097, 256)])
def test_quantize_ragged_row_counts(M, K):
    bits = workloads.activations(M, K, "student_t3", M + K, 0.005, 50.0)
    q, s = gpu_quantize(bits)
    assert_quant_equal(bits, q, s, f"ragged {M}x{K}")


def _act_inputs():
    seen = {}
    for wl in workloads.WORKLOADS.values():
        for lin in wl.linears:
            key = (lin.M, lin.K, lin.x_dist, lin.x_seed, lin.outlier_frac, lin.outlier_factor)
            seen.setdefault(key, lin)
    return list(seen.values())


@pytest.mark.parametrize("lin", _act_inputs(), ids=lambda l: f"{l.name}-{l.M}x{l.K}")
def test_quantize_full_workload_activations(lin):
    say("quantize full", lin.name, lin.M, lin.K)
    bits = lin.make_x()
    q, s = gpu_quantize(bits)
    assert_quant_equal(bits, q, s, lin.name)


@pytest.mark.parametrize("lin", [l for wl in workloads.WORKLOADS.values() for l in wl.linears],
                         ids=lambda l: f"{l.name}-W{l.N}x{l.K}")
def test_pack_weight_full_workloads(lin):
    say("pack weight", lin.name, lin.N, lin.K)
    bits = lin.make_w()
    q, s = gpu_quantize(bits, weight=True)
    assert_quant_equal(bits, q, s, lin.name + " weight")


# ---------------------------------------------------------------------------
# exact accumulators
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("M,N,K", [(1, 1, 64), (3, 5, 128), (16, 16, 64), (257, 255, 192),
                                   (300, 520, 1024), (256, 256, 3072), (513, 1000, 640),
                                   (1, 4099, 128), (2049, 3, 320)])
def test_gemm_i32_random_codes(M, N, K):
    say("gemm i32", M, N, K)
    qx = rand_packed(M, K, seed=M * 7 + K)
    qw = rand_packed(N, K, seed=N * 11 + K)
    acc = jq.jq_w4a4_gemm_i32(torch.from_numpy(qx).cuda(), torch.from_numpy(qw).cuda())
    torch.cuda.synchronize()
    ref = oracle.w4a4_gemm_i32(qx, qw)
    bad = np.argwhere(acc.cpu().numpy() != ref)
    assert bad.size == 0, f"{len(bad)} accumulators differ, first {bad[:4].tolist()}"


# Many tiles (more than one round of blocks), ragged M and N, short and
# medium K; both tile heights of the int8 GEMM (a CPU test checks that).
MANY_TILES = [(4096, 8192, 384), (2100, 9000, 512), (300, 70000, 512), (2049, 3, 384),
              (4608, 4096, 1152), (9216, 3072, 640), (33, 4099, 1536), (4090, 8192, 384)]


@pytest.mark.parametrize("M,N,K", MANY_TILES)
def test_gemm_i32_many_tiles(M, N, K):
    say("gemm i32 many tiles", M, N, K)
    qx = rand_packed(M, K, seed=M * 5 + K)
    qw = rand_packed(N, K, seed=N * 3 + K)
    acc = jq.jq_w4a4_gemm_i32(torch.from_numpy(qx).cuda(), torch.from_numpy(qw).cuda())
    torch.cuda.synchronize()
    ref = oracle.w4a4_gemm_i32(qx, qw)
    bad = np.argwhere(acc.cpu().numpy() != ref)
    assert bad.size == 0, f"{len(bad)} accumulators differ, first {bad[:4].tolist()}"


@pytest.mark.parametrize("code_x,code_w", [(-8, -8), (7, -8), (-7, 7)])
def test_gemm_i32_extreme_codes_max_k(code_x, code_w):
    K = 65536
    M, N = 300, 260
    nib = lambda c: (c & 0xF) | ((c & 0xF) << 4)
    qx = np.full((M, K // 2), nib(code_x), np.uint8)
    qw = np.full((N, K // 2), nib(code_w), np.uint8)
    acc = jq.jq_w4a4_gemm_i32(torch.from_numpy(qx).cuda(), torch.from_numpy(qw).cuda()).cpu().numpy()
    assert np.all(acc == code_x * code_w * K)


# ---------------------------------------------------------------------------
# whole layer
# ---------------------------------------------------------------------------


def _layer(bits_x, bits_w, bits_b):
    x = dev_bf16(bits_x)
    wq, sw = jq.jq_pack_weight_int4(dev_bf16(bits_w))
    b = None if bits_b is None else dev_bf16(bits_b)
    y = jq.jq_w4a4_linear(x, wq, sw, b)
    torch.cuda.synchronize()
    return jq.bf16_bits(y), wq.cpu().numpy(), sw.cpu().numpy()


@pytest.mark.parametrize("with_bias", [False, True])
def test_linear_tiny_workload_full(with_bias):
    lin = workloads.WORKLOADS["tiny"].linears[0]
    x, w = lin.make_x(), lin.make_w()
    b = workloads.bias(lin.N, 0.01, 2) if with_bias else None
    y, wq, sw = _layer(x, w, b)
    rq, rs = oracle.pack_weight_int4(w)
    assert np.array_equal(wq, rq) and np.array_equal(sw.view(np.uint32), rs.view(np.uint32))
    ref = oracle.w4a4_linear(x, rq, rs, b)
    assert_bf16_close(y, ref, f"tiny bias={with_bias}")


RAGGED_LINEARS = [(77, 3072, 130, True), (1, 64, 1, False), (5, 192, 4096, True), (300, 1088, 260, False),
                  (513, 256, 777, True), (513, 1024, 777, True), (300, 6912, 777, True), (2048, 6912, 520, False),
                  (4100, 384, 2050, True), (4090, 384, 12288, True)]


@pytest.mark.parametrize("M,K,N,bias", RAGGED_LINEARS)
def test_linear_ragged(M, K, N, bias):
    say("linear ragged", M, K, N, bias)
    x = workloads.activations(M, K, "student_t3", M + 3, 0.01, 50.0)
    w = workloads.weights(N, K, 0.02, N + 5)
    b = workloads.bias(N, 0.01, 7) if bias else None
    y, wq, sw = _layer(x, w, b)
    ref = oracle.w4a4_linear(x, wq, sw, b)
    assert_bf16_close(y, ref, f"ragged {M}x{K}->{N}")


def test_linear_edge_rows_outputs():
    """Zero, subnormal, huge and tie rows through the whole layer."""
    K, N = 256, 96
    x = _edge_rows(K, seed=5)
    w = workloads.weights(N, K, 0.02, 6)
    b = workloads.bias(N, 0.01, 7)
    y, wq, sw = _layer(x, w, b)
    ref = oracle.w4a4_linear(x, wq, sw, b)
    assert_bf16_close(y, ref, "edge rows")
    y0, _, _ = _layer(x, w, None)
    assert_bf16_close(y0, oracle.w4a4_linear(x, wq, sw, None), "edge rows no bias")


def _sample_rows(M, n=40, seed=0):
    rng = np.random.default_rng(seed)
    fixed = [0, 1, 255, 256, M // 2, M - 257, M - 2, M - 1]
    rows = set(r for r in fixed if 0 <= r < M)
    rows.update(rng.integers(0, M, size=n).tolist())
    return np.array(sorted(rows))


def test_shared_quantization_matches_linear():
    """Gate and up projections of the 8B block share one activation quantisation."""
    wl = workloads.WORKLOADS["dllm_block"]
    gate, up = wl.linears[0], wl.linears[1]
    M = 512
    x_bits = gate.make_x()[:M]
    x = dev_bf16(x_bits)
    q, s = jq.jq_quantize_act(x)
    for lin in (gate, up):
        w_bits = lin.make_w()[:1024]
        wq, sw = jq.jq_pack_weight_int4(dev_bf16(w_bits))
        y1 = jq.jq_w4a4_gemm(q, s, wq, sw)
        y2 = jq.jq_w4a4_linear(x, wq, sw)
        torch.cuda.synchronize()
        assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


def test_determinism_and_side_stream():
    lin = workloads.WORKLOADS["attn_proj"].linears[0]
    x_bits = lin.make_x()[:1024]
    w_bits = lin.make_w()[:768]
    x = dev_bf16(x_bits)
    wq, sw = jq.jq_pack_weight_int4(dev_bf16(w_bits))
    y1 = jq.jq_w4a4_linear(x, wq, sw)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        y2 = jq.jq_w4a4_linear(x, wq, sw)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    ref = oracle.w4a4_linear(x_bits, wq.cpu().numpy(), sw.cpu().numpy())
    assert_bf16_close(jq.bf16_bits(y1), ref, "side stream")
