"""The allocation-free BF6 linear (jq_w4a4_f6_linear_noalloc) against the
workspace one (jq_w4a4_f6_linear) through the C ABI: bit-identical outputs on
two calls in a row, the second with a smaller input (so its scratch still
holds the first call's larger operand), and the size limit.  Runs last: it
shares the library's per-device scratch with nothing else in the suite.
"""

import numpy as np
import pytest
import torch

from paper_2609_33601_amd import jq, workloads

pytestmark = pytest.mark.gpu


def _prepare(lin, bias_bits=None):
    x = jq.bf16_tensor(lin.make_x(), "cuda")
    wq, sw = jq.jq_pack_weight_int4(jq.bf16_tensor(lin.make_w(), "cuda"))
    wf6 = jq.jq_int4_to_f6_weight(wq)
    b = None if bias_bits is None else jq.bf16_tensor(bias_bits, "cuda")
    return x, wf6, sw, b


def _ragged(M, K, N, seed):
    return workloads.Linear("ragged", M=M, K=K, N=N, x_dist="student_t3", x_seed=seed,
                            outlier_frac=0.005, outlier_factor=50.0, w_std=0.02, w_seed=seed + 1)


def _same(a, b):
    return int((a.view(torch.int16) != b.view(torch.int16)).sum())


def test_noalloc_matches_workspace_linear_on_two_calls():
    jq.lib()
    big = workloads.WORKLOADS["mlp_down"].linears[0]  # 9216 x 12288 -> 3072: 81 MiB of scratch
    assert jq.jq_w4a4_f6_workspace_bytes(big.M, big.K) <= jq.JQ_NOALLOC_SCRATCH_BYTES
    small = _ragged(777, 1088, 520, 40)  # ragged tiles, K = 64 mod 128, with bias
    small_bias = workloads.bias(small.N, 0.01, 42)
    print(f"noalloc: call 1 {big.M}x{big.K}->{big.N}, call 2 {small.M}x{small.K}->{small.N} (bias)", flush=True)
    xa, wa, sa, _ = _prepare(big)
    xb, wb, sb, bb = _prepare(small, small_bias)
    ya = jq.jq_w4a4_f6_linear_noalloc(xa, wa, sa)
    yb = jq.jq_w4a4_f6_linear_noalloc(xb, wb, sb, bb)
    torch.cuda.synchronize()
    ra = jq.jq_w4a4_f6_linear(xa, wa, sa)
    rb = jq.jq_w4a4_f6_linear(xb, wb, sb, bb)
    torch.cuda.synchronize()
    assert _same(ya, ra) == 0
    assert _same(yb, rb) == 0
    # the same again in the other order, on the scratch left by the calls above
    yb2 = jq.jq_w4a4_f6_linear_noalloc(xb, wb, sb, bb)
    ya2 = jq.jq_w4a4_f6_linear_noalloc(xa, wa, sa)
    torch.cuda.synchronize()
    assert _same(yb2, rb) == 0 and _same(ya2, ra) == 0


def test_noalloc_small_case_matches_oracle():
    import oracle

    lin = workloads.WORKLOADS["tiny"].linears[0]
    b_bits = workloads.bias(lin.N, 0.01, 2)
    x, wf6, sw, b = _prepare(lin, b_bits)
    y = jq.jq_w4a4_f6_linear_noalloc(x, wf6, sw, b)
    torch.cuda.synchronize()
    rq, rs = oracle.pack_weight_int4(lin.make_w())
    ref = oracle.w4a4_linear(lin.make_x(), rq, rs, b_bits)
    assert np.array_equal(jq.bf16_bits(y), ref)


def test_noalloc_refuses_inputs_beyond_its_scratch():
    lin = _ragged(9216, 16384, 256, 50)  # 108 MiB of operand: more than the scratch holds
    assert jq.jq_w4a4_f6_workspace_bytes(lin.M, lin.K) > jq.JQ_NOALLOC_SCRATCH_BYTES
    x = torch.zeros((lin.M, lin.K), dtype=torch.bfloat16, device="cuda")
    wf6 = torch.zeros((jq.jq_f6_operand_bytes(lin.N, lin.K),), dtype=torch.uint8, device="cuda")
    sw = torch.ones((lin.N,), dtype=torch.float32, device="cuda")
    y = torch.full((lin.M, lin.N), 7.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(jq.JQError) as e:
        jq.jq_w4a4_f6_linear_noalloc(x, wf6, sw, y=y)
    assert e.value.status == jq.JQ_ERR_WORKSPACE_TOO_SMALL
    torch.cuda.synchronize()
    assert bool((y == 7.0).all()), "a refused call wrote its output"
