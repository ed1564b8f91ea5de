"""Full-size parity against the oracle: every code, scale, accumulator and output.

For every linear of the workloads (the tiny one, the DiT attention projection
and fused QKV, the FLUX-12B MLP-up and MLP-down for one and for two images,
the four 8B diffusion-LLM block linears) at its full size, the oracle computes
the whole layer on the host: the per-token codes and scales, the exact
accumulators of every output and the bf16 outputs.  The GPU computes the same
layer on both engines exactly as the benchmark launches it
(jq_w4a4_linear, jq_w4a4_f6_linear; for W1.58A4 jq_w158a4_linear and
jq_w4a4_f6_linear on the re-encoded ternary weight), and the accumulators
through jq_w4a4_gemm_i32 / jq_w158a4_gemm_i32 / jq_w4a4_f6_gemm_i32 from the
quantised activations the layer left in its own workspace.

Bar: zero differing codes, scales, accumulators and bf16 outputs over the
whole tensors (the stated tolerance is one bf16 ulp on outputs; the kernels
follow the oracle's rounding sequence, so they are expected to be, and are
required here to be, bit-identical).
"""

import os
import sys

import numpy as np
import pytest

import oracle
from paper_2609_33601_amd import jq, workloads
from tests.test_gpu_f6 import decode_f6

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

LINEARS = [l for wl in workloads.WORKLOADS.values() for l in wl.linears]
WS_ALIGN = 256


def say(*a):
    print("[gpu-full]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the parity tests need an MI355X")
    if not os.path.exists(jq.LIB_PATH):
        pytest.fail("libjq.so is not built")
    yield
    _ACT.clear()
    torch.cuda.synchronize()


# activations and their oracle quantisation, shared by the W4A4 and W1.58A4
# tests of a linear (and by linears that share their input)
_ACT = {}


def _activations(lin):
    key = (lin.M, lin.K, lin.x_dist, lin.x_seed, lin.outlier_frac, lin.outlier_factor)
    if key not in _ACT:
        x_bits = lin.make_x()
        _ACT.clear()  # keep one input at a time in host memory
        _ACT[key] = (x_bits, *oracle.quantize_act(x_bits))
    return _ACT[key]


def _round_up(v, a=WS_ALIGN):
    return (v + a - 1) // a * a


def _count_diff(a, b):
    a, b = np.asarray(a), np.asarray(b)
    assert a.shape == b.shape, (a.shape, b.shape)
    return int(np.count_nonzero(a != b))


def _assert_f6_codes(xf6_host, packed_ref, M, K, what):
    """Decode the BF6 activation operand band by band and compare every code
    (padding included, which must be zero) with the oracle's."""
    codes = oracle.unpack_int4(packed_ref).astype(np.int64)
    ks = 2 * ((K + 127) // 128)
    band_bytes = ks * 1536
    nb = (M + 31) // 32
    Kp = 128 * ((K + 127) // 128)
    step = 16
    bad = 0
    for b0 in range(0, nb, step):
        b1 = min(nb, b0 + step)
        got = decode_f6(xf6_host[b0 * band_bytes:b1 * band_bytes], (b1 - b0) * 32, K)
        ref = np.zeros(((b1 - b0) * 32, Kp), np.int64)
        r1 = min(M, b1 * 32)
        ref[: r1 - b0 * 32, :K] = codes[b0 * 32:r1]
        bad += _count_diff(got, ref)
    assert bad == 0, f"{what}: {bad} BF6 codes differ from the oracle's"


def _gpu_int8(x, w_dev, b, M, K, ternary):
    """The layer on the int8 engine through its linear entry point, and the
    accumulators from the codes left in its workspace."""
    if ternary:
        wq, sw = jq.jq_pack_weight_ternary(w_dev)
    else:
        wq, sw = jq.jq_pack_weight_int4(w_dev)
    ws = torch.empty(jq.jq_w4a4_workspace_bytes(M, K), dtype=torch.uint8, device="cuda")
    lin_fn = jq.jq_w158a4_linear if ternary else jq.jq_w4a4_linear
    y = lin_fn(x, wq, sw, b, workspace=ws)
    qx = ws[: M * K // 2].view(M, K // 2)
    sx = ws[_round_up(M * K // 2): _round_up(M * K // 2) + 4 * M].view(torch.float32)
    acc = (jq.jq_w158a4_gemm_i32 if ternary else jq.jq_w4a4_gemm_i32)(qx, wq)
    return wq, sw, y, qx, sx, acc


def _gpu_bf6(x, wq, sw, b, M, K, N, ternary):
    """The same layer on the BF6 engine (weights re-encoded once), and the
    accumulators from the BF6 operand left in its workspace."""
    wf6 = (jq.jq_ternary_to_f6_weight if ternary else jq.jq_int4_to_f6_weight)(wq)
    ws = torch.empty(jq.jq_w4a4_f6_workspace_bytes(M, K), dtype=torch.uint8, device="cuda")
    y = jq.jq_w4a4_f6_linear(x, wf6, sw, b, workspace=ws)
    nbytes = jq.jq_f6_operand_bytes(M, K)
    xf6 = ws[:nbytes]
    sx = ws[_round_up(nbytes): _round_up(nbytes) + 4 * M].view(torch.float32)
    acc = jq.jq_w4a4_f6_gemm_i32(xf6, M, K, wf6, N)
    return y, xf6, sx, acc


def _check_layer(lin, ternary):
    M, K, N = lin.M, lin.K, lin.N
    layer = "W1.58A4" if ternary else "W4A4"
    say(f"{layer} {lin.name} {M}x{K}->{N}: oracle")
    x_bits, rqx, rsx = _activations(lin)
    w_bits, b_bits = lin.make_w(), lin.make_bias()
    if ternary:
        rw, rsw = oracle.pack_weight_ternary(w_bits)
        acc_ref = oracle.code_gemm(oracle.unpack_int4(rqx), oracle.unpack_ternary(rw))
    else:
        rw, rsw = oracle.pack_weight_int4(w_bits)
        acc_ref = oracle.code_gemm(oracle.unpack_int4(rqx), oracle.unpack_int4(rw))
    y_ref = oracle.epilogue(acc_ref, rsx, rsw, b_bits)
    acc_ref = acc_ref.astype(np.int32)  # |acc| <= 64 K < 2^31

    say(f"{layer} {lin.name}: int8 engine")
    x = jq.bf16_tensor(x_bits, "cuda")
    b = None if b_bits is None else jq.bf16_tensor(b_bits, "cuda")
    wq, sw, y4, qx, sx4, acc4 = _gpu_int8(x, jq.bf16_tensor(w_bits, "cuda"), b, M, K, ternary)
    torch.cuda.synchronize()
    assert _count_diff(wq.cpu().numpy(), rw) == 0, "weight codes differ"
    assert _count_diff(sw.cpu().numpy().view(np.uint32), rsw.view(np.uint32)) == 0, "weight scales differ"
    assert _count_diff(qx.cpu().numpy(), rqx) == 0, "activation codes differ"
    assert _count_diff(sx4.cpu().numpy().view(np.uint32), rsx.view(np.uint32)) == 0, "activation scales differ"
    d = _count_diff(acc4.cpu().numpy(), acc_ref)
    assert d == 0, f"int8 engine: {d} of {M * N} accumulators differ"
    d = _count_diff(jq.bf16_bits(y4), y_ref)
    assert d == 0, f"int8 engine: {d} of {M * N} outputs differ"
    del acc4, y4, qx, sx4

    say(f"{layer} {lin.name}: bf6 engine")
    y6, xf6, sx6, acc6 = _gpu_bf6(x, wq, sw, b, M, K, N, ternary)
    torch.cuda.synchronize()
    assert _count_diff(sx6.cpu().numpy().view(np.uint32), rsx.view(np.uint32)) == 0, "bf6 activation scales differ"
    _assert_f6_codes(xf6.cpu().numpy(), rqx, M, K, f"{lin.name} bf6 operand")
    d = _count_diff(acc6.cpu().numpy(), acc_ref)
    assert d == 0, f"bf6 engine: {d} of {M * N} accumulators differ"
    d = _count_diff(jq.bf16_bits(y6), y_ref)
    assert d == 0, f"bf6 engine: {d} of {M * N} outputs differ"
    say(f"{layer} {lin.name}: {M * N} outputs and accumulators equal on both engines")


@pytest.mark.parametrize("lin,ternary", [(l, t) for l in LINEARS for t in (False, True)],
                         ids=lambda v: ("W1.58A4" if v else "W4A4") if isinstance(v, bool)
                         else f"{v.name}-{v.M}x{v.K}x{v.N}")
def test_full_size_every_output(lin, ternary):
    _check_layer(lin, ternary)
