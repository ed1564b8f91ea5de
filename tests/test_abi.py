"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects bad arguments before launching anything.

Only argument-validation paths are exercised here (fake device addresses are
never dereferenced because every call below fails validation first).
"""

import ctypes
import os
import re

import pytest

from paper_2609_33601_amd import jq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "jq.h")

pytestmark = pytest.mark.skipif(not os.path.exists(jq.LIB_PATH),
                                reason="libjq.so not built (run __graft_entry__.build())")

A = 0x10000  # a fake, 256-byte-aligned address
MIS = A + 2  # 2-byte aligned only


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(jq_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = header_functions()
    assert len(names) == 36, names
    lib = ctypes.CDLL(jq.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), f"libjq.so does not export {n}"
    assert set(names) == set(jq.SIGNATURES), "binding and header disagree"


def test_status_strings_and_version():
    assert jq.jq_status_string(0) == "JQ_OK"
    assert jq.jq_status_string(4) == "JQ_ERR_WORKSPACE_TOO_SMALL"
    assert jq.jq_status_string(99) == "JQ_ERR_UNKNOWN"
    assert jq.jq_version() >= 100


def test_workspace_bytes():
    L = jq.lib()
    assert L.jq_w4a4_workspace_bytes(4608, 3072) == 4608 * 1536 + 18432
    assert L.jq_w4a4_workspace_bytes(1, 64) == 256 + 256
    assert L.jq_w4a4_workspace_bytes(3, 128) == 256 + 256
    assert L.jq_w4a4_workspace_bytes(0, 64) == 0
    assert L.jq_w4a4_workspace_bytes(8, 100) == 0


@pytest.mark.parametrize("fn", ["jq_quantize_act", "jq_pack_weight_int4", "jq_pack_weight_ternary"])
def test_quantize_validation(fn):
    f = getattr(jq.lib(), fn)
    assert f(None, 8, 64, A, A, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, 8, 64, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, 8, 64, A, None, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, 0, 64, A, A, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, -3, 64, A, A, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, 8, 0, A, A, None) == jq.JQ_ERR_INVALID_ARG
    for K in (2, 32, 100, 65536 + 64):
        assert f(A, 8, K, A, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE, K
    assert f(A, 1 << 31, 64, A, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert f(MIS, 8, 64, A, A, None) == jq.JQ_ERR_MISALIGNED
    assert f(A, 8, 64, A + 8, A, None) == jq.JQ_ERR_MISALIGNED
    assert f(A, 8, 64, A, A + 1, None) == jq.JQ_ERR_MISALIGNED


@pytest.mark.parametrize("fn", ["jq_w4a4_linear", "jq_w158a4_linear"])
def test_linear_validation(fn):
    f = getattr(jq.lib(), fn)
    need = jq.lib().jq_w4a4_workspace_bytes(16, 128)
    ok = dict(x=A, M=16, K=128, wq=A, sw=A, N=32, b=None, y=A, ws=A, wsb=need, s=None)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(a["x"], a["M"], a["K"], a["wq"], a["sw"], a["N"], a["b"], a["y"], a["ws"], a["wsb"], a["s"])

    for k in ("x", "wq", "sw", "y", "ws"):
        assert call(**{k: None}) == jq.JQ_ERR_INVALID_ARG, k
    assert call(M=0) == jq.JQ_ERR_INVALID_ARG
    assert call(N=0) == jq.JQ_ERR_INVALID_ARG
    assert call(K=96) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert call(x=MIS) == jq.JQ_ERR_MISALIGNED
    assert call(wq=A + 4) == jq.JQ_ERR_MISALIGNED
    assert call(y=A + 8) == jq.JQ_ERR_MISALIGNED
    assert call(sw=A + 2) == jq.JQ_ERR_MISALIGNED
    assert call(b=A + 1) == jq.JQ_ERR_MISALIGNED
    assert call(ws=A + 16) == jq.JQ_ERR_MISALIGNED
    assert call(wsb=need - 1) == jq.JQ_ERR_WORKSPACE_TOO_SMALL
    assert call(wsb=0) == jq.JQ_ERR_WORKSPACE_TOO_SMALL


@pytest.mark.parametrize("fmt", ["w4a4", "w158a4"])
def test_gemm_validation(fmt):
    g = getattr(jq.lib(), f"jq_{fmt}_gemm")
    assert g(None, A, 4, 64, A, A, 4, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert g(A, None, 4, 64, A, A, 4, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert g(A, A, 4, 64, A, None, 4, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert g(A, A, 4, 64, A, A, 4, None, None, None) == jq.JQ_ERR_INVALID_ARG
    assert g(A, A, 4, 192 + 32, A, A, 4, None, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert g(A + 8, A, 4, 64, A, A, 4, None, A, None) == jq.JQ_ERR_MISALIGNED
    i = getattr(jq.lib(), f"jq_{fmt}_gemm_i32")
    assert i(None, 4, 64, A, 4, A, None) == jq.JQ_ERR_INVALID_ARG
    assert i(A, 4, 64, A, 4, None, None) == jq.JQ_ERR_INVALID_ARG
    assert i(A, 4, 64, A, -1, A, None) == jq.JQ_ERR_INVALID_ARG
    assert i(A, 4, 48, A, 4, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert i(A, 4, 64, A, 4, A + 4, None) == jq.JQ_ERR_MISALIGNED
    assert i(A, 1 << 30, 64, A, 1 << 20, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert i(A, 1 << 20, 4096, A, 64, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE  # 2 GiB packed activations
    # 2 GiB packed weights: N*K/2 bytes for int4, N*K/4 for ternary
    big_n = (1 << 16) if fmt == "w4a4" else (1 << 17)
    assert i(A, 64, 65536, A, big_n, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE


def test_group_workspace_bytes():
    L = jq.lib()
    assert L.jq_w4a4g_workspace_bytes(4608, 3072, 64) == 4608 * 1536 + 4608 * 48 * 4
    assert L.jq_w4a4g_workspace_bytes(1, 128, 128) == 256 + 256
    assert L.jq_w4a4g_workspace_bytes(8, 192, 128) == 0   # K % G != 0
    assert L.jq_w4a4g_workspace_bytes(8, 128, 32) == 0    # unsupported group size
    assert L.jq_w4a4g_workspace_bytes(0, 128, 64) == 0


@pytest.mark.parametrize("fn", ["jq_quantize_act_group", "jq_pack_weight_int4_group"])
def test_group_quantize_validation(fn):
    f = getattr(jq.lib(), fn)
    assert f(None, 8, 128, 64, A, A, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, 8, 128, 64, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, 8, 128, 64, A, None, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, 0, 128, 64, A, A, None) == jq.JQ_ERR_INVALID_ARG
    for K, G in ((192, 128), (128, 32), (128, 0), (128, 256), (100, 64)):
        assert f(A, 8, K, G, A, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE, (K, G)
    assert f(A, 1 << 30, 65536, 64, A, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert f(MIS, 8, 128, 64, A, A, None) == jq.JQ_ERR_MISALIGNED
    assert f(A, 8, 128, 64, A + 8, A, None) == jq.JQ_ERR_MISALIGNED
    assert f(A, 8, 128, 64, A, A + 2, None) == jq.JQ_ERR_MISALIGNED


def test_group_gemm_validation():
    L = jq.lib()
    g, f32 = L.jq_w4a4g_gemm, L.jq_w4a4g_gemm_f32
    for k in range(5):
        args = [A, A, 4, 128, 64, A, A, 4, None, A, None]
        args[[0, 1, 5, 6, 9][k]] = None
        assert g(*args) == jq.JQ_ERR_INVALID_ARG, k
    assert g(A, A, 4, 192, 128, A, A, 4, None, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert g(A, A, 4, 128, 64, A, A, 4, A + 1, A, None) == jq.JQ_ERR_MISALIGNED
    assert g(A, A + 2, 4, 128, 64, A, A, 4, None, A, None) == jq.JQ_ERR_MISALIGNED
    assert f32(A, A, 4, 128, 64, A, A, 4, None, None) == jq.JQ_ERR_INVALID_ARG
    assert f32(A, A, 4, 128, 64, A, A, 4, A + 8, None) == jq.JQ_ERR_MISALIGNED
    assert f32(A, A, 1 << 20, 4096, 64, A, A, 64, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    lin = L.jq_w4a4g_linear
    need = L.jq_w4a4g_workspace_bytes(16, 128, 64)
    assert lin(A, 16, 128, 64, A, A, 32, None, A, A, need - 1, None) == jq.JQ_ERR_WORKSPACE_TOO_SMALL
    assert lin(A, 16, 128, 64, A, A, 32, None, A, A + 16, need, None) == jq.JQ_ERR_MISALIGNED
    assert lin(A, 16, 128, 64, A, A, 32, None, A, None, need, None) == jq.JQ_ERR_INVALID_ARG
    assert lin(A, 16, 192, 128, A, A, 32, None, A, A, need, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(jq, "_lib", None)
    monkeypatch.setattr(jq, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        jq.lib()


# ---------------------------------------------------------------------------
# BF6 engine


def test_f6_sizes():
    L = jq.lib()
    # ceil(rows/32) bands x 2*ceil(K/128) k-steps x 1536 bytes
    assert L.jq_f6_operand_bytes(9216, 12288) == 288 * 192 * 1536
    assert L.jq_f6_operand_bytes(1, 64) == 1 * 2 * 1536
    assert L.jq_f6_operand_bytes(33, 192) == 2 * 4 * 1536
    assert L.jq_f6_operand_bytes(0, 64) == 0
    assert L.jq_f6_operand_bytes(8, 96) == 0
    assert L.jq_w4a4_f6_workspace_bytes(4608, 3072) == 144 * 48 * 1536 + 18432
    assert L.jq_w4a4_f6_workspace_bytes(1, 64) == 3072 + 256
    assert L.jq_w4a4_f6_workspace_bytes(5, 100) == 0


def test_f6_quantize_and_convert_validation():
    L = jq.lib()
    assert L.jq_quantize_act_f6(None, 8, 64, A, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_quantize_act_f6(A, 0, 64, A, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_quantize_act_f6(A, 8, 96, A, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert L.jq_quantize_act_f6(A, 8, 65600, A, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert L.jq_quantize_act_f6(MIS, 8, 64, A, A, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_quantize_act_f6(A, 8, 64, MIS, A, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_int4_to_f6(None, 8, 64, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_int4_to_f6(A, 8, 64, None, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_int4_to_f6(A, -1, 64, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_int4_to_f6(A, 8, 32, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert L.jq_int4_to_f6(A, 8, 64, MIS, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_int4_to_f6_weight(None, 8, 64, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_int4_to_f6_weight(A, 8, 64, None, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_int4_to_f6_weight(A, 0, 64, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_int4_to_f6_weight(A, 8, 96, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert L.jq_int4_to_f6_weight(MIS, 8, 64, A, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_ternary_to_f6_weight(None, 8, 64, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_ternary_to_f6_weight(A, 8, 64, None, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_ternary_to_f6_weight(A, 0, 64, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_ternary_to_f6_weight(A, 8, 96, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert L.jq_ternary_to_f6_weight(MIS, 8, 64, A, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_ternary_to_f6_weight(A, 8, 64, MIS, None) == jq.JQ_ERR_MISALIGNED


def test_f6_gemm_and_linear_validation():
    L = jq.lib()
    ws = L.jq_w4a4_f6_workspace_bytes(8, 64)
    assert L.jq_w4a4_f6_linear(None, 8, 64, A, A, 8, None, A, A, ws, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_w4a4_f6_linear(A, 8, 64, A, A, 8, None, A, None, ws, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_w4a4_f6_linear(A, 8, 64, A, A, 8, None, A, A, ws - 1, None) == jq.JQ_ERR_WORKSPACE_TOO_SMALL
    assert L.jq_w4a4_f6_linear(A, 8, 64, A, A, 8, None, A, A + 16, ws, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_w4a4_f6_linear(A, 8, 64, MIS, A, 8, None, A, A, ws, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_w4a4_f6_linear(A, 8, 64, A, A, 8, A + 1, A, A, ws, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_w4a4_f6_gemm(A, None, 8, 64, A, A, 8, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_w4a4_f6_gemm(A, A, 8, 160, A, A, 8, None, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert L.jq_w4a4_f6_gemm(A, A, 8, 64, A, A, 0, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_w4a4_f6_gemm(A, A, 8, 64, A, A, 8, None, MIS, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_w4a4_f6_gemm_i32(None, 8, 64, A, 8, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_w4a4_f6_gemm_i32(A, 8, 64, A, 8, None, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_w4a4_f6_gemm_i32(A, 8, 64, A, 8, MIS, None) == jq.JQ_ERR_MISALIGNED
    # operands of 2 GiB or more are refused (31-bit buffer descriptors)
    assert L.jq_w4a4_f6_gemm_i32(A, 1 << 22, 65536, A, 8, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE


def test_f6_quantize_batch_validation():
    # argument checks of the batched BF6 quantiser, all before anything is launched
    f = jq.lib().jq_quantize_act_f6_batch
    P = ctypes.c_void_p * 2
    I = ctypes.c_int64 * 2

    def call(n=2, x=(A, A), M=(8, 16), K=(64, 128), q=(A, A), s=(A, A)):
        return f(n, P(*x), I(*M), I(*K), P(*q), P(*s), None)

    assert call(n=0) == jq.JQ_ERR_INVALID_ARG
    assert call(n=9) == jq.JQ_ERR_INVALID_ARG
    assert f(2, None, I(8, 8), I(64, 64), P(A, A), P(A, A), None) == jq.JQ_ERR_INVALID_ARG
    assert call(x=(A, None)) == jq.JQ_ERR_INVALID_ARG
    assert call(q=(None, A)) == jq.JQ_ERR_INVALID_ARG
    assert call(s=(A, None)) == jq.JQ_ERR_INVALID_ARG
    assert call(M=(8, 0)) == jq.JQ_ERR_INVALID_ARG
    assert call(K=(64, 96)) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert call(K=(65600, 64)) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert call(x=(A, MIS)) == jq.JQ_ERR_MISALIGNED
    assert call(q=(A + 8, A)) == jq.JQ_ERR_MISALIGNED
    assert call(s=(A, A + 2)) == jq.JQ_ERR_MISALIGNED


def test_f6_linear_noalloc_validation():
    # argument checks of the allocation-free linear, all before the scratch is looked up
    L = jq.lib()
    f = L.jq_w4a4_f6_linear_noalloc
    assert f(None, 8, 64, A, A, 8, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, 8, 64, None, A, 8, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, 8, 64, A, None, 8, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, 8, 64, A, A, 8, None, None, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, 0, 64, A, A, 8, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert f(A, 8, 96, A, A, 8, None, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert f(MIS, 8, 64, A, A, 8, None, A, None) == jq.JQ_ERR_MISALIGNED
    assert f(A, 8, 64, A, A, 8, A + 1, A, None) == jq.JQ_ERR_MISALIGNED
    # the largest input the scratch holds, and the first beyond it
    assert jq.JQ_NOALLOC_SCRATCH_BYTES == 96 << 20
    assert L.jq_w4a4_f6_workspace_bytes(9216, 12288) <= jq.JQ_NOALLOC_SCRATCH_BYTES
    assert L.jq_w4a4_f6_workspace_bytes(9216, 16384) > jq.JQ_NOALLOC_SCRATCH_BYTES
    assert f(A, 9216, 16384, A, A, 8, None, A, None) == jq.JQ_ERR_WORKSPACE_TOO_SMALL
    assert f(A, 1 << 20, 128, A, A, 8, None, A, None) == jq.JQ_ERR_WORKSPACE_TOO_SMALL


def test_group_f6_validation():
    L = jq.lib()
    # workspace: BF6 operand + scales, each rounded up to 256 bytes; 0 for invalid sizes
    assert L.jq_w4a4g_f6_workspace_bytes(8, 128, 64) == L.jq_f6_operand_bytes(8, 128) + 256
    assert L.jq_w4a4g_f6_workspace_bytes(8, 128, 32) == 0
    assert L.jq_w4a4g_f6_workspace_bytes(8, 192, 128) == 0
    assert L.jq_quantize_act_group_f6(None, 8, 128, 64, A, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_quantize_act_group_f6(A, 8, 128, 96, A, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert L.jq_quantize_act_group_f6(A, 8, 192, 128, A, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert L.jq_quantize_act_group_f6(A, 8, 128, 64, MIS, A, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_quantize_act_group_f6(A, 8, 128, 64, A, A + 1, None) == jq.JQ_ERR_MISALIGNED
    ws = L.jq_w4a4g_f6_workspace_bytes(8, 128, 64)
    assert L.jq_w4a4g_f6_linear(None, 8, 128, 64, A, A, 8, None, A, A, ws, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_w4a4g_f6_linear(A, 8, 128, 64, A, A, 8, None, A, A, ws - 1, None) == jq.JQ_ERR_WORKSPACE_TOO_SMALL
    assert L.jq_w4a4g_f6_linear(A, 8, 128, 64, A, A, 8, None, A, A + 16, ws, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_w4a4g_f6_linear(A, 8, 128, 64, A, None, 8, None, A, A, ws, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_w4a4g_f6_gemm(A, None, 8, 128, 64, A, A, 8, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_w4a4g_f6_gemm(A, A, 8, 128, 48, A, A, 8, None, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE
    assert L.jq_w4a4g_f6_gemm(A, A, 8, 128, 64, A, A, 0, None, A, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_w4a4g_f6_gemm(A, A, 8, 128, 64, A, A, 8, A + 1, A, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_w4a4g_f6_gemm(A, A, 8, 128, 64, MIS, A, 8, None, A, None) == jq.JQ_ERR_MISALIGNED
    assert L.jq_w4a4g_f6_gemm_f32(A, A, 8, 128, 64, A, A, 8, None, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_w4a4g_f6_gemm_f32(A, A, 8, 128, 64, A, A, 8, MIS, None) == jq.JQ_ERR_MISALIGNED
    # operands of 2 GiB or more are refused (31-bit buffer descriptors)
    assert L.jq_w4a4g_f6_gemm_f32(A, A, 1 << 22, 65536, 64, A, A, 8, A, None) == jq.JQ_ERR_UNSUPPORTED_SHAPE


def test_gemm_plan():
    """The int8 GEMM's tile height: 112 rows where 128-row tiles would leave
    the last round of blocks mostly empty and 112-row tiles fill it, else 128."""
    plan = lambda M, N, K: jq.jq_gemm_plan(M, N, K, 256)
    assert plan(9216, 3072, 12288) == 112   # FLUX MLP-down: 864 tiles -> 996 (two full rounds of 512)
    assert plan(4608, 3072, 12288) == 112   # FLUX MLP-down, one image: 432 -> 504 of 512 slots
    assert plan(4608, 12288, 3072) == 128   # FLUX MLP-up: the last 128-row round is three-eighths full
    assert plan(4608, 3072, 3072) == 112    # DiT attention projection
    assert plan(4608, 9216, 3072) == 112    # DiT fused QKV
    assert plan(4096, 12288, 4096) == 128   # dLLM gate/up: whole rounds
    assert plan(4096, 4096, 12288) == 128   # dLLM down
    assert plan(4096, 4096, 4096) == 128    # dLLM o-proj
    assert plan(8192, 4096, 12288) == 128   # whole rounds
    assert plan(64, 256, 256) in (112, 128)
    L = jq.lib()
    t = ctypes.c_int()
    assert L.jq_gemm_plan(8, 8, 64, 0, ctypes.byref(t)) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_gemm_plan(8, 8, 64, 256, None) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_gemm_plan(0, 8, 64, 256, ctypes.byref(t)) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_gemm_plan(8, 8, 96, 256, ctypes.byref(t)) == jq.JQ_ERR_UNSUPPORTED_SHAPE


def test_gpu_parity_shapes_cover_both_int8_tile_heights():
    """The GPU parity cases run the int8 GEMM at both tile heights, with M
    ragged against each (the height is chosen per shape by the library)."""
    from tests.test_gpu_parity import MANY_TILES, RAGGED_LINEARS

    plan = lambda M, N, K: jq.jq_gemm_plan(M, N, K, 256)
    gemm = {plan(M, N, K) for M, N, K in MANY_TILES}
    layer = {plan(M, N, K) for M, K, N, _ in RAGGED_LINEARS}
    assert gemm == {112, 128} and layer == {112, 128}
    for rows in (112, 128):
        assert any(plan(M, N, K) == rows and M % rows for M, N, K in MANY_TILES), rows
        assert any(plan(M, N, K) == rows and M % rows for M, K, N, _ in RAGGED_LINEARS), rows


def test_f6_gemm_plan():
    """The BF6 GEMM's block shape: one 8-wave block per CU where 256-row tiles
    cover M evenly or K is long, two 4-wave blocks (128-row tiles) otherwise."""
    plan = lambda M, N, K: jq.jq_f6_gemm_plan(M, N, K, 256)
    assert plan(4608, 12288, 3072) == (4, 128)    # FLUX MLP-up: 224-row tiles would not cover M evenly
    assert plan(9216, 3072, 12288) == (8, 224)    # FLUX MLP-down: long K
    assert plan(4096, 12288, 4096) == (8, 256)    # dLLM gate/up: 256-row tiles fit exactly
    assert plan(4096, 4096, 12288) == (8, 256)    # dLLM down
    assert plan(4608, 3072, 3072) == (4, 128)     # DiT attention projection
    assert plan(4608, 3072, 8192) == (8, 224)     # K above 6144 keeps the 8-wave block
    assert plan(64, 256, 256) == (4, 128)         # small shapes
    L = jq.lib()
    w, t = ctypes.c_int(), ctypes.c_int()
    assert L.jq_f6_gemm_plan(8, 8, 64, 0, ctypes.byref(w), ctypes.byref(t)) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_f6_gemm_plan(8, 8, 64, 256, None, ctypes.byref(t)) == jq.JQ_ERR_INVALID_ARG
    assert L.jq_f6_gemm_plan(8, 8, 96, 256, ctypes.byref(w), ctypes.byref(t)) == jq.JQ_ERR_UNSUPPORTED_SHAPE
