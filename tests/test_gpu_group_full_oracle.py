"""Full-size group-wise parity against the oracle: every code, scale, group sum and output.

For every group-wise workload layer (FLUX-12B MLP-up and MLP-down in groups
of 64; the DiT attention projection, the fused QKV and the four 8B
diffusion-LLM block linears in groups of 128) the oracle quantises the whole
activation and weight tensors per group, computes the fp32 group sums of
every output through its compiled form (oracle/group_sum.c, equal bit for bit
to the numpy oracle by the CPU tests) and rounds them to bf16 with the bias.
The GPU computes the same layer on both engines exactly as the benchmark
launches it (jq_w4a4g_linear, jq_w4a4g_f6_linear), and the group sums through
jq_w4a4g_gemm_f32 / jq_w4a4g_f6_gemm_f32 from the operands the layer left in
its own workspace.

Bar: zero differing codes, scales, fp32 group sums and bf16 outputs over the
whole tensors (the kernels take the oracle's rounding sequence step for step).
"""

import sys

import numpy as np
import pytest

import oracle
from oracle import group_sum_c
from paper_2609_33601_amd import jq, workloads
from tests.test_gpu_full_oracle import _assert_f6_codes, _count_diff, _round_up

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

LAYERS = [(workloads.WORKLOADS[n].linears[0], 64) for n in ("mlp_up", "mlp_down")] + \
         [(workloads.WORKLOADS[n].linears[0], 128) for n in ("attn_proj", "qkv")] + \
         [(l, 128) for l in workloads.WORKLOADS["dllm_block"].linears]


def say(*a):
    print("[gpu-group-full]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _ready():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible: the parity tests need an MI355X")
    group_sum_c.lib()  # raises if the compiled oracle is not built
    yield
    torch.cuda.synchronize()


def _bits_equal(got_f32, ref_f32, what, total):
    d = _count_diff(got_f32.view(np.uint32), ref_f32.view(np.uint32))
    assert d == 0, f"{what}: {d} of {total} differ"


@pytest.mark.parametrize("lin,G", LAYERS, ids=lambda v: f"{v.name}-{v.M}x{v.K}x{v.N}" if hasattr(v, "name")
                         else f"G{v}")
def test_group_full_size_every_output(lin, G):
    M, K, N = lin.M, lin.K, lin.N
    say(f"group{G} {lin.name} {M}x{K}->{N}: oracle")
    x_bits, w_bits, b_bits = lin.make_x(), lin.make_w(), lin.make_bias()
    rwq, rsw = oracle.pack_weight_int4_group(w_bits, G)
    rqx, rsx = oracle.quantize_act_group(x_bits, G)
    S_ref = group_sum_c.w4a4g_gemm_f32(rqx, rsx, rwq, rsw, G)
    y_ref = oracle.group_epilogue(S_ref, b_bits)

    say(f"group{G} {lin.name}: int8 engine")
    x = jq.bf16_tensor(x_bits, "cuda")
    b = None if b_bits is None else jq.bf16_tensor(b_bits, "cuda")
    wq, sw = jq.jq_pack_weight_int4_group(jq.bf16_tensor(w_bits, "cuda"), G)
    ws = torch.empty(jq.jq_w4a4g_workspace_bytes(M, K, G), dtype=torch.uint8, device="cuda")
    y4 = jq.jq_w4a4g_linear(x, wq, sw, G, b, workspace=ws)
    codes = M * K // 2
    qx = ws[:codes].view(M, K // 2)
    sx = ws[_round_up(codes): _round_up(codes) + 4 * M * (K // G)].view(torch.float32).view(M, K // G)
    S4 = jq.jq_w4a4g_gemm_f32(qx, sx, wq, sw, G)
    torch.cuda.synchronize()
    assert _count_diff(wq.cpu().numpy(), rwq) == 0, "weight codes differ"
    _bits_equal(sw.cpu().numpy(), rsw, "weight group scales", rsw.size)
    assert _count_diff(qx.cpu().numpy(), rqx) == 0, "activation codes differ"
    _bits_equal(sx.cpu().numpy(), rsx, "activation group scales", rsx.size)
    _bits_equal(S4.cpu().numpy(), S_ref, "int8 engine group sums", M * N)
    d = _count_diff(jq.bf16_bits(y4), y_ref)
    assert d == 0, f"int8 engine: {d} of {M * N} outputs differ"
    del y4, S4, qx, sx, ws

    say(f"group{G} {lin.name}: bf6 engine")
    wf6 = jq.jq_int4_to_f6_weight(wq)
    ws6 = torch.empty(jq.jq_w4a4g_f6_workspace_bytes(M, K, G), dtype=torch.uint8, device="cuda")
    y6 = jq.jq_w4a4g_f6_linear(x, wf6, sw, G, b, workspace=ws6)
    nbytes = jq.jq_f6_operand_bytes(M, K)
    xf6 = ws6[:nbytes]
    sx6 = ws6[_round_up(nbytes): _round_up(nbytes) + 4 * M * (K // G)].view(torch.float32).view(M, K // G)
    S6 = jq.jq_w4a4g_f6_gemm_f32(xf6, sx6, wf6, sw, G)
    torch.cuda.synchronize()
    _bits_equal(sx6.cpu().numpy(), rsx, "bf6 activation group scales", rsx.size)
    _assert_f6_codes(xf6.cpu().numpy(), rqx, M, K, f"{lin.name} bf6 operand")
    _bits_equal(S6.cpu().numpy(), S_ref, "bf6 engine group sums", M * N)
    d = _count_diff(jq.bf16_bits(y6), y_ref)
    assert d == 0, f"bf6 engine: {d} of {M * N} outputs differ"
    say(f"group{G} {lin.name}: {M * N} outputs and group sums equal on both engines")
