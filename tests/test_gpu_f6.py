"""GPU parity of the BF6 engine (the W4A4 layer on the 6-bit matrix cores)
through the C ABI, against the CPU oracle.

Bars, as for the packed-int4 path: scales, codes and int32 accumulators
bit-exact; bf16 outputs within 1 bf16 ulp of the oracle (expected
bit-identical).  The codes inside a BF6 operand are read back with a decoder of
the layout documented in include/jq.h, written here from that description.
At full workload sizes every output and accumulator is compared with the
oracle in tests/test_gpu_full_oracle.py.
"""

import os
import sys

import numpy as np
import pytest

import oracle
from paper_2609_33601_amd import jq, workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def say(*a):
    print("[gpu-f6]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the parity tests need an MI355X")
    if not os.path.exists(jq.LIB_PATH):
        pytest.fail("libjq.so is not built")
    yield
    torch.cuda.synchronize()


# ---------------------------------------------------------------------------
# BF6 operand decoder (test side)
# ---------------------------------------------------------------------------


def _e3m2_table():
    t = np.zeros(64, np.float64)
    for e in range(64):
        sign = -1.0 if e & 0x20 else 1.0
        ex, m = (e >> 2) & 7, e & 3
        t[e] = sign * ((m / 4) * 2.0 ** -2 if ex == 0 else (1 + m / 4) * 2.0 ** (ex - 3))
    return t


E3M2 = _e3m2_table()


def decode_f6(buf, rows, K):
    """BF6 operand bytes -> integer codes [32*ceil(rows/32), 128*ceil(K/128)]."""
    KS = 2 * ((K + 127) // 128)
    NB = (rows + 31) // 32
    frag = np.asarray(buf, np.uint8).reshape(NB, KS, 1536)
    lane = np.concatenate([frag[:, :, :1024].reshape(NB, KS, 64, 16),
                           frag[:, :, 1024:].reshape(NB, KS, 64, 8)], axis=3)   # 24 bytes per lane
    bits = np.unpackbits(lane, axis=3, bitorder="little").reshape(NB, KS, 64, 32, 6)
    fields = (bits * (1 << np.arange(6))).sum(axis=4)
    vals = E3M2[fields]                                                         # [NB, KS, L, p]
    assert np.all(vals == np.round(vals)), "non-integer BF6 value"
    codes = vals.astype(np.int64).reshape(NB, KS, 2, 32, 32)                    # [b, s, h, r, p]
    codes = codes.transpose(0, 3, 1, 2, 4).reshape(NB * 32, KS * 64)            # row 32b + r, k 64s + 32h + p
    return codes


def decode_f6_weight(buf, rows, K):
    """BF6 operand bytes in the weight layout -> integer codes, as decode_f6."""
    KS = 2 * ((K + 127) // 128)
    NB = (rows + 31) // 32
    blk = np.asarray(buf, np.uint8).reshape(NB, KS // 2, 3, 64, 16)              # [b, u, plane, L, 16]
    lane = blk.transpose(0, 1, 3, 2, 4).reshape(NB, KS // 2, 64, 48)              # 48 bytes per lane
    lane = lane.reshape(NB, KS // 2, 64, 2, 24).transpose(0, 1, 3, 2, 4)          # [b, u, t, L, 24]
    bits = np.unpackbits(lane, axis=4, bitorder="little").reshape(NB, KS // 2, 2, 64, 32, 6)
    fields = (bits * (1 << np.arange(6))).sum(axis=5)
    vals = E3M2[fields]
    assert np.all(vals == np.round(vals)), "non-integer BF6 value"
    codes = vals.astype(np.int64).reshape(NB, KS, 2, 32, 32)                      # k-step s = 2u + t
    return codes.transpose(0, 3, 1, 2, 4).reshape(NB * 32, KS * 64)


def padded_codes(packed, rows, K):
    c = oracle.unpack_int4(packed).astype(np.int64)
    out = np.zeros((32 * ((rows + 31) // 32), 128 * ((K + 127) // 128)), np.int64)
    out[:rows, :K] = c
    return out


def dev_bf16(bits):
    return jq.bf16_tensor(bits, "cuda")


def rand_packed(rows, K, seed):
    return np.random.default_rng(seed).integers(0, 256, size=(rows, K // 2), dtype=np.uint8)


def ulp_bf16(v):
    a = np.abs(v)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a >= 2.0 ** -126, np.exp2(e - 7), 2.0 ** -133)


def assert_bf16_close(y_bits, ref_bits, what):
    y = oracle.bf16_bits_to_f32(y_bits).astype(np.float64)
    r = oracle.bf16_bits_to_f32(ref_bits).astype(np.float64)
    fin = np.isfinite(r)
    assert np.array_equal(y_bits[~fin], ref_bits[~fin]), f"{what}: non-finite outputs differ"
    err = np.where(fin, np.abs(np.where(fin, y, 0) - np.where(fin, r, 0)), 0)
    bad = np.argwhere(err > ulp_bf16(np.where(fin, r, 1.0)))
    assert bad.size == 0, f"{what}: {len(bad)} outputs beyond 1 bf16 ulp, first {bad[:4].tolist()}"
    say(f"{what}: bit-identical fraction {np.mean(y_bits == ref_bits):.6f}")


def _edge_rows(K, seed):
    from tests.test_gpu_parity import _edge_rows as edge

    return edge(K, seed)


# ---------------------------------------------------------------------------
# decoder self-check on a hand-built fragment (no GPU involved)
# ---------------------------------------------------------------------------


def test_decoder_hand_built_fragment():
    # one band, K = 128 (two k-steps); lane 5 of k-step 1 = row 5, codes 64..95
    enc = {0: 0x00, 1: 0x0C, 2: 0x10, 3: 0x12, 4: 0x14, 5: 0x15, 6: 0x16, 7: 0x17, 8: 0x18}
    codes = [(p % 16) - 8 for p in range(32)]
    word = 0
    for p, c in enumerate(codes):
        word |= (enc[abs(c)] | (0x20 if c < 0 else 0)) << (6 * p)
    lane_bytes = word.to_bytes(24, "little")
    buf = np.zeros(2 * 1536, np.uint8)
    base = 1536 + 0  # fragment (band 0, k-step 1)
    buf[base + 16 * 5: base + 16 * 5 + 16] = np.frombuffer(lane_bytes[:16], np.uint8)
    buf[base + 1024 + 8 * 5: base + 1024 + 8 * 5 + 8] = np.frombuffer(lane_bytes[16:], np.uint8)
    dec = decode_f6(buf, 32, 128)
    assert dec[5, 64:96].tolist() == codes
    dec[5, 64:96] = 0
    assert not dec.any()


def test_weight_decoder_hand_built_pair():
    # weight layout, one band, K = 256: k-step 3 = the second k-step of pair
    # u = 1; lane 37 = row 5, half 1: codes 3*64 + 32 .. +31 of row 5
    enc = {0: 0x00, 1: 0x0C, 2: 0x10, 3: 0x12, 4: 0x14, 5: 0x15, 6: 0x16, 7: 0x17, 8: 0x18}
    codes = [7 - (p % 16) for p in range(32)]
    word = 0
    for p, c in enumerate(codes):
        word |= (enc[abs(c)] | (0x20 if c < 0 else 0)) << (6 * p)
    d = word.to_bytes(24, "little")             # dwords d0..d5 of the group
    buf = np.zeros(4 * 1536, np.uint8)
    base, L = 3072, 37
    # lane bytes 24..47 of the pair record: the last 8 bytes of plane 1, all of plane 2
    buf[base + 1024 + 16 * L + 8: base + 1024 + 16 * L + 16] = np.frombuffer(d[:8], np.uint8)
    buf[base + 2048 + 16 * L: base + 2048 + 16 * L + 16] = np.frombuffer(d[8:], np.uint8)
    dec = decode_f6_weight(buf, 32, 256)
    assert dec[5, 224:256].tolist() == codes
    dec[5, 224:256] = 0
    assert not dec.any()


# ---------------------------------------------------------------------------
# quantiser and converter
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("M,K,src", [(64, 256, "tiny"), (16, 256, "edge"), (16, 4160, "edge"),
                                     (77, 192, "t"), (33, 3072, "t"), (5, 12288, "t"), (40, 16384, "edge"),
                                     (3, 20480, "t"), (2, 65536, "t")])
def test_quantize_f6_matches_oracle(M, K, src):
    if src == "tiny":
        bits = workloads.WORKLOADS["tiny"].linears[0].make_x()
    elif src == "edge":
        bits = _edge_rows(K, seed=K)
        M = bits.shape[0]
    else:
        bits = workloads.activations(M, K, "student_t3", M + K, 0.01, 50.0)
    say("quantize f6", M, K, src)
    xf6, s = jq.jq_quantize_act_f6(dev_bf16(bits))
    torch.cuda.synchronize()
    rq, rs = oracle.quantize_act(bits)
    assert np.array_equal(s.cpu().numpy().view(np.uint32), rs.view(np.uint32)), "scales differ"
    got = decode_f6(xf6.cpu().numpy(), M, K)
    bad = np.argwhere(got != padded_codes(rq, M, K))
    assert bad.size == 0, f"{len(bad)} codes differ, first {bad[:4].tolist()}"


@pytest.mark.parametrize("rows,K", [(1, 64), (31, 128), (33, 192), (100, 4160), (64, 12288)])
def test_int4_to_f6_lossless(rows, K):
    q = rand_packed(rows, K, seed=rows * 3 + K)
    f6 = jq.jq_int4_to_f6(torch.from_numpy(q).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(decode_f6(f6.cpu().numpy(), rows, K), padded_codes(q, rows, K))


@pytest.mark.parametrize("rows,K", [(1, 64), (31, 128), (33, 192), (100, 4160), (64, 12288)])
def test_int4_to_f6_weight_lossless(rows, K):
    q = rand_packed(rows, K, seed=rows * 5 + K)
    f6 = jq.jq_int4_to_f6_weight(torch.from_numpy(q).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(decode_f6_weight(f6.cpu().numpy(), rows, K), padded_codes(q, rows, K))


# ---------------------------------------------------------------------------
# exact accumulators
# ---------------------------------------------------------------------------


def f6_i32(qx, qw):
    M, N, K = qx.shape[0], qw.shape[0], 2 * qx.shape[1]
    xf6 = jq.jq_int4_to_f6(torch.from_numpy(qx).cuda())
    wf6 = jq.jq_int4_to_f6_weight(torch.from_numpy(qw).cuda())
    acc = jq.jq_w4a4_f6_gemm_i32(xf6, M, K, wf6, N)
    torch.cuda.synchronize()
    return acc.cpu().numpy()


@pytest.mark.parametrize("M,N,K", [(1, 1, 64), (3, 5, 128), (32, 32, 64), (257, 255, 192),
                                   (300, 520, 1024), (256, 256, 3072), (513, 1000, 640),
                                   (1, 4099, 128), (2049, 3, 320), (512, 768, 12288),
                                   (300, 777, 6912), (2048, 2048, 7680)])
def test_f6_gemm_i32_random_codes(M, N, K):
    say("f6 gemm i32", M, N, K)
    qx = rand_packed(M, K, seed=M * 7 + K)
    qw = rand_packed(N, K, seed=N * 11 + K)
    got = f6_i32(qx, qw)
    ref = oracle.w4a4_gemm_i32(qx, qw)
    bad = np.argwhere(got != ref)
    assert bad.size == 0, f"{len(bad)} accumulators differ, first {bad[:4].tolist()}"


@pytest.mark.parametrize("M,N,K", [(4096, 8192, 384), (2100, 9000, 448), (4608, 4096, 256), (300, 70000, 512),
                                   (2100, 9000, 6912), (4096, 8192, 6912)])
def test_f6_gemm_i32_several_tiles_per_block(M, N, K):
    """More tiles than CUs: blocks walk several tiles, with loads running
    ahead across tile boundaries (three or more stages per tile), or one tile
    each (fewer than three stages)."""
    say("f6 gemm i32 many tiles", M, N, K)
    qx = rand_packed(M, K, seed=M + 2 * K)
    qw = rand_packed(N, K, seed=N + 3 * K)
    got = f6_i32(qx, qw)
    ref = oracle.w4a4_gemm_i32(qx, qw)
    bad = np.argwhere(got != ref)
    assert bad.size == 0, f"{len(bad)} accumulators differ, first {bad[:4].tolist()}"


@pytest.mark.parametrize("code_x,code_w", [(-8, -8), (7, -8), (-7, 7)])
def test_f6_gemm_i32_extreme_codes_max_k(code_x, code_w):
    K, M, N = 65536, 300, 260
    say("f6 gemm extreme", code_x, code_w)
    nib = lambda c: (c & 0xF) | ((c & 0xF) << 4)
    qx = np.full((M, K // 2), nib(code_x), np.uint8)
    qw = np.full((N, K // 2), nib(code_w), np.uint8)
    assert np.all(f6_i32(qx, qw) == code_x * code_w * K)


def test_f6_gemm_i32_large_partial_sums_then_small_terms():
    """A large accumulator followed by +-1 products: exact only if no low bits are dropped."""
    K, M, N = 16384, 64, 64
    cx = np.full((M, K), 7, np.int64)
    cw = np.full((N, K), 7, np.int64)
    rng = np.random.default_rng(3)
    cx[:, K // 2:] = rng.choice([-1, 0, 1], size=(M, K // 2))
    cw[:, K // 2:] = rng.choice([-1, 1], size=(N, K // 2))
    qx, qw = oracle.pack_int4(cx), oracle.pack_int4(cw)
    assert np.array_equal(f6_i32(qx, qw), oracle.w4a4_gemm_i32(qx, qw))


# ---------------------------------------------------------------------------
# whole layer
# ---------------------------------------------------------------------------


def f6_layer(bits_x, bits_w, bits_b):
    x = dev_bf16(bits_x)
    wq, sw = jq.jq_pack_weight_int4(dev_bf16(bits_w))
    wf6 = jq.jq_int4_to_f6_weight(wq)
    b = None if bits_b is None else dev_bf16(bits_b)
    y = jq.jq_w4a4_f6_linear(x, wf6, sw, b)
    torch.cuda.synchronize()
    return jq.bf16_bits(y), wq.cpu().numpy(), sw.cpu().numpy()


@pytest.mark.parametrize("with_bias", [False, True])
def test_f6_linear_tiny_workload(with_bias):
    lin = workloads.WORKLOADS["tiny"].linears[0]
    x, w = lin.make_x(), lin.make_w()
    b = workloads.bias(lin.N, 0.01, 2) if with_bias else None
    y, wq, sw = f6_layer(x, w, b)
    rq, rs = oracle.pack_weight_int4(w)
    assert np.array_equal(wq, rq) and np.array_equal(sw.view(np.uint32), rs.view(np.uint32))
    assert_bf16_close(y, oracle.w4a4_linear(x, rq, rs, b), f"f6 tiny bias={with_bias}")


@pytest.mark.parametrize("M,K,N,bias", [(77, 3072, 130, True), (1, 64, 1, False), (5, 192, 4096, True),
                                        (300, 1088, 260, False), (513, 256, 777, True), (257, 4160, 300, True),
                                        (300, 6912, 777, True), (513, 7680, 1000, True), (2048, 6912, 520, False)])
def test_f6_linear_ragged(M, K, N, bias):
    say("f6 linear ragged", M, K, N, bias)
    x = workloads.activations(M, K, "student_t3", M + 3, 0.01, 50.0)
    w = workloads.weights(N, K, 0.02, N + 5)
    b = workloads.bias(N, 0.01, 7) if bias else None
    y, wq, sw = f6_layer(x, w, b)
    assert_bf16_close(y, oracle.w4a4_linear(x, wq, sw, b), f"f6 ragged {M}x{K}->{N}")


def test_f6_linear_edge_rows():
    K, N = 256, 96
    x = _edge_rows(K, seed=5)
    w = workloads.weights(N, K, 0.02, 6)
    b = workloads.bias(N, 0.01, 7)
    y, wq, sw = f6_layer(x, w, b)
    assert_bf16_close(y, oracle.w4a4_linear(x, wq, sw, b), "f6 edge rows")


def test_f6_gemm_matches_linear():
    """GEMM on a separately quantised operand equals the whole linear."""
    lin = workloads.WORKLOADS["dllm_block"].linears[0]
    M = 512
    x = dev_bf16(lin.make_x()[:M])
    wq, sw = jq.jq_pack_weight_int4(dev_bf16(lin.make_w()[:1024]))
    wf6 = jq.jq_int4_to_f6_weight(wq)
    xf6, s = jq.jq_quantize_act_f6(x)
    y1 = jq.jq_w4a4_f6_gemm(xf6, s, lin.K, wf6, sw)
    y2 = jq.jq_w4a4_f6_linear(x, wf6, sw)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


# ---------------------------------------------------------------------------
# W1.58A4 on the BF6 engine: ternary codes in the BF6 weight layout
# ---------------------------------------------------------------------------


def rand_ternary(rows, K, seed):
    return np.random.default_rng(seed).integers(-1, 2, size=(rows, K)).astype(np.int8)


@pytest.mark.parametrize("rows,K", [(1, 64), (31, 128), (33, 192), (100, 4160), (64, 12288)])
def test_ternary_to_f6_weight_lossless(rows, K):
    t = rand_ternary(rows, K, seed=rows * 3 + K)
    f6 = jq.jq_ternary_to_f6_weight(torch.from_numpy(oracle.pack_ternary(t)).cuda())
    torch.cuda.synchronize()
    ref = np.zeros((32 * ((rows + 31) // 32), 128 * ((K + 127) // 128)), np.int64)
    ref[:rows, :K] = t
    assert np.array_equal(decode_f6_weight(f6.cpu().numpy(), rows, K), ref)


@pytest.mark.parametrize("M,N,K", [(3, 5, 128), (257, 255, 192), (2100, 9000, 448), (512, 768, 12288)])
def test_f6_w158a4_gemm_i32_random_codes(M, N, K):
    say("f6 ternary gemm i32", M, N, K)
    qx = rand_packed(M, K, seed=M * 13 + K)
    wt = oracle.pack_ternary(rand_ternary(N, K, seed=N * 17 + K))
    xf6 = jq.jq_int4_to_f6(torch.from_numpy(qx).cuda())
    wf6 = jq.jq_ternary_to_f6_weight(torch.from_numpy(wt).cuda())
    acc = jq.jq_w4a4_f6_gemm_i32(xf6, M, K, wf6, N)
    torch.cuda.synchronize()
    ref = oracle.w158a4_gemm_i32(qx, wt)
    bad = np.argwhere(acc.cpu().numpy() != ref)
    assert bad.size == 0, f"{len(bad)} accumulators differ, first {bad[:4].tolist()}"


def f6_ternary_layer(x_bits, w_bits, b_bits):
    """The W1.58A4 layer on the BF6 engine and on the int8 engine, same inputs."""
    x = dev_bf16(x_bits)
    wt, g = jq.jq_pack_weight_ternary(dev_bf16(w_bits))
    wf6 = jq.jq_ternary_to_f6_weight(wt)
    b = None if b_bits is None else dev_bf16(b_bits)
    y6 = jq.jq_w4a4_f6_linear(x, wf6, g, b)
    y8 = jq.jq_w158a4_linear(x, wt, g, b)
    torch.cuda.synchronize()
    return y6, y8, wt.cpu().numpy(), g.cpu().numpy()


@pytest.mark.parametrize("M,K,N,bias", [(77, 3072, 130, True), (1, 64, 1, False), (513, 256, 777, True),
                                        (257, 4160, 300, True)])
def test_f6_w158a4_linear_ragged(M, K, N, bias):
    say("f6 ternary linear ragged", M, K, N, bias)
    x = workloads.activations(M, K, "student_t3", M + 7, 0.01, 50.0)
    w = workloads.weights(N, K, 0.02, N + 9)
    b = workloads.bias(N, 0.01, 11) if bias else None
    y6, y8, wt, g = f6_ternary_layer(x, w, b)
    assert torch.equal(y6.view(torch.int16), y8.view(torch.int16))
    assert_bf16_close(jq.bf16_bits(y6), oracle.w158a4_linear(x, wt, g, b), f"f6 ternary {M}x{K}->{N}")


# ---------------------------------------------------------------------------
# Batched BF6 quantiser: several independent inputs in one call
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("shapes", [
    [(4608, 3072), (9216, 12288)],                                  # the FLUX MLP pair
    [(1, 64), (33, 192), (4097, 256), (7, 16384), (5, 20480)],      # ragged rows; the last row is past 16384 codes
    [(100 + 37 * i, 64 * (1 + 7 * i)) for i in range(8)],          # eight inputs
    [(64, 4160)],                                                   # one input
], ids=["flux_pair", "ragged_and_long", "eight", "single"])
def test_quantize_f6_batch_matches_single_launches(shapes):
    say("f6 quantise batch", shapes)
    bits = [workloads.activations(M, K, "student_t3", 70 + i, 0.005, 50.0) for i, (M, K) in enumerate(shapes)]
    xs = [dev_bf16(b) for b in bits]
    qb, sb = jq.jq_quantize_act_f6_batch(xs)
    torch.cuda.synchronize()
    for i, (x, (M, K)) in enumerate(zip(xs, shapes)):
        q1, s1 = jq.jq_quantize_act_f6(x)
        torch.cuda.synchronize()
        assert torch.equal(qb[i], q1), f"input {i} {M}x{K}: BF6 operand differs from its own launch"
        assert torch.equal(sb[i].view(torch.int32), s1.view(torch.int32)), f"input {i}: scales differ"
        if M * K <= 1 << 22:
            rq, rs = oracle.quantize_act(bits[i])
            assert np.array_equal(sb[i].cpu().numpy().view(np.uint32), rs.view(np.uint32))
            assert np.array_equal(decode_f6(qb[i].cpu().numpy(), M, K), padded_codes(rq, M, K)), f"input {i}: codes"


def test_quantize_f6_batch_outputs_feed_the_gemm():
    """The FLUX MLP pair quantised in one call, then each linear's GEMM: the
    outputs equal the whole layer's (jq_w4a4_f6_linear) bit for bit."""
    lins = workloads.FLUX_MLP.linears
    xs, ws, bs = [], [], []
    for lin in lins:
        xs.append(dev_bf16(lin.make_x()))
        wq, sw = jq.jq_pack_weight_int4(dev_bf16(lin.make_w()))
        ws.append((jq.jq_int4_to_f6_weight(wq), sw))
        b = lin.make_bias()
        bs.append(None if b is None else dev_bf16(b))
    qs, ss = jq.jq_quantize_act_f6_batch(xs)
    for lin, x, (wf6, sw), b, q, s in zip(lins, xs, ws, bs, qs, ss):
        y1 = jq.jq_w4a4_f6_gemm(q, s, lin.K, wf6, sw, b)
        y2 = jq.jq_w4a4_f6_linear(x, wf6, sw, b)
        torch.cuda.synchronize()
        assert torch.equal(y1.view(torch.int16), y2.view(torch.int16)), lin.name
