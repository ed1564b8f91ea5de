"""Python binding of libjq (include/jq.h): argument marshalling only.

Every function takes torch tensors that live on the GPU, passes their device
pointers and the current HIP stream to the C ABI, and raises JQError on a
non-OK status.  All arithmetic happens in the HIP kernels; if libjq.so is not
built, every call raises instead of computing anything another way.
"""

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libjq.so")

JQ_OK = 0
JQ_ERR_INVALID_ARG = 1
JQ_ERR_UNSUPPORTED_SHAPE = 2
JQ_ERR_MISALIGNED = 3
JQ_ERR_WORKSPACE_TOO_SMALL = 4
JQ_ERR_HIP = 5

# Symbols the library exports, with (restype, argtypes).
_vp, _i64, _sz, _fp, _ip = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p
SIGNATURES = {
    "jq_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "jq_version": (ctypes.c_int, []),
    "jq_quantize_act": (ctypes.c_int, [_vp, _i64, _i64, _vp, _fp, _vp]),
    "jq_pack_weight_int4": (ctypes.c_int, [_vp, _i64, _i64, _vp, _fp, _vp]),
    "jq_w4a4_workspace_bytes": (_sz, [_i64, _i64]),
    "jq_w4a4_linear": (ctypes.c_int, [_vp, _i64, _i64, _vp, _fp, _i64, _vp, _vp, _vp, _sz, _vp]),
    "jq_w4a4_gemm": (ctypes.c_int, [_vp, _fp, _i64, _i64, _vp, _fp, _i64, _vp, _vp, _vp]),
    "jq_w4a4_gemm_i32": (ctypes.c_int, [_vp, _i64, _i64, _vp, _i64, _ip, _vp]),
    "jq_pack_weight_ternary": (ctypes.c_int, [_vp, _i64, _i64, _vp, _fp, _vp]),
    "jq_w158a4_linear": (ctypes.c_int, [_vp, _i64, _i64, _vp, _fp, _i64, _vp, _vp, _vp, _sz, _vp]),
    "jq_w158a4_gemm": (ctypes.c_int, [_vp, _fp, _i64, _i64, _vp, _fp, _i64, _vp, _vp, _vp]),
    "jq_w158a4_gemm_i32": (ctypes.c_int, [_vp, _i64, _i64, _vp, _i64, _ip, _vp]),
    "jq_quantize_act_group": (ctypes.c_int, [_vp, _i64, _i64, _i64, _vp, _fp, _vp]),
    "jq_pack_weight_int4_group": (ctypes.c_int, [_vp, _i64, _i64, _i64, _vp, _fp, _vp]),
    "jq_w4a4g_workspace_bytes": (_sz, [_i64, _i64, _i64]),
    "jq_w4a4g_linear": (ctypes.c_int, [_vp, _i64, _i64, _i64, _vp, _fp, _i64, _vp, _vp, _vp, _sz, _vp]),
    "jq_w4a4g_gemm": (ctypes.c_int, [_vp, _fp, _i64, _i64, _i64, _vp, _fp, _i64, _vp, _vp, _vp]),
    "jq_w4a4g_gemm_f32": (ctypes.c_int, [_vp, _fp, _i64, _i64, _i64, _vp, _fp, _i64, _fp, _vp]),
    "jq_f6_operand_bytes": (_sz, [_i64, _i64]),
    "jq_quantize_act_f6": (ctypes.c_int, [_vp, _i64, _i64, _vp, _fp, _vp]),
    "jq_quantize_act_f6_batch": (ctypes.c_int, [ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _vp]),
    "jq_int4_to_f6": (ctypes.c_int, [_vp, _i64, _i64, _vp, _vp]),
    "jq_int4_to_f6_weight": (ctypes.c_int, [_vp, _i64, _i64, _vp, _vp]),
    "jq_ternary_to_f6_weight": (ctypes.c_int, [_vp, _i64, _i64, _vp, _vp]),
    "jq_w4a4_f6_workspace_bytes": (_sz, [_i64, _i64]),
    "jq_w4a4_f6_linear": (ctypes.c_int, [_vp, _i64, _i64, _vp, _fp, _i64, _vp, _vp, _vp, _sz, _vp]),
    "jq_w4a4_f6_linear_noalloc": (ctypes.c_int, [_vp, _i64, _i64, _vp, _fp, _i64, _vp, _vp, _vp]),
    "jq_w4a4_f6_gemm": (ctypes.c_int, [_vp, _fp, _i64, _i64, _vp, _fp, _i64, _vp, _vp, _vp]),
    "jq_w4a4_f6_gemm_i32": (ctypes.c_int, [_vp, _i64, _i64, _vp, _i64, _ip, _vp]),
    "jq_f6_gemm_plan": (ctypes.c_int, [_i64, _i64, _i64, ctypes.c_int, _ip, _ip]),
    "jq_gemm_plan": (ctypes.c_int, [_i64, _i64, _i64, ctypes.c_int, _ip]),
    "jq_quantize_act_group_f6": (ctypes.c_int, [_vp, _i64, _i64, _i64, _vp, _fp, _vp]),
    "jq_w4a4g_f6_workspace_bytes": (ctypes.c_size_t, [_i64, _i64, _i64]),
    "jq_w4a4g_f6_linear": (ctypes.c_int, [_vp, _i64, _i64, _i64, _vp, _fp, _i64, _vp, _vp, _vp, _sz, _vp]),
    "jq_w4a4g_f6_gemm": (ctypes.c_int, [_vp, _fp, _i64, _i64, _i64, _vp, _fp, _i64, _vp, _vp, _vp]),
    "jq_w4a4g_f6_gemm_f32": (ctypes.c_int, [_vp, _fp, _i64, _i64, _i64, _vp, _fp, _i64, _fp, _vp]),
}

_lib = None


class JQError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {jq_status_string(status)} ({status})")


def lib():
    """The loaded libjq.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build the HIP library first "
                "(python -c 'import __graft_entry__ as g; g.build()')")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(l, name)
            fn.restype = res
            fn.argtypes = args
        _lib = l
    return _lib


def jq_status_string(status):
    return lib().jq_status_string(int(status)).decode()


def jq_version():
    return lib().jq_version()


def _check(status, where):
    if status != JQ_OK:
        raise JQError(status, where)


def _torch():
    import torch

    return torch


def _stream_ptr(stream):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t, dtype, shape, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU, got {t.device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def jq_w4a4_workspace_bytes(M, K):
    return int(lib().jq_w4a4_workspace_bytes(int(M), int(K)))


def jq_quantize_act(x, q=None, scale=None, stream=None):
    """x bf16 [M,K] -> (q uint8 [M,K/2], scale fp32 [M])."""
    torch = _torch()
    M, K = x.shape
    if q is None:
        q = torch.empty((M, K // 2), dtype=torch.uint8, device=x.device)
    if scale is None:
        scale = torch.empty((M,), dtype=torch.float32, device=x.device)
    st = lib().jq_quantize_act(_dev(x, torch.bfloat16, None, "x"), M, K,
                               _dev(q, torch.uint8, (M, K // 2), "q"),
                               _dev(scale, torch.float32, (M,), "scale"), _stream_ptr(stream))
    _check(st, "jq_quantize_act")
    return q, scale


def jq_pack_weight_int4(w, wq=None, w_scale=None, stream=None):
    """w bf16 [N,K] -> (wq uint8 [N,K/2], w_scale fp32 [N])."""
    torch = _torch()
    N, K = w.shape
    if wq is None:
        wq = torch.empty((N, K // 2), dtype=torch.uint8, device=w.device)
    if w_scale is None:
        w_scale = torch.empty((N,), dtype=torch.float32, device=w.device)
    st = lib().jq_pack_weight_int4(_dev(w, torch.bfloat16, None, "w"), N, K,
                                   _dev(wq, torch.uint8, (N, K // 2), "wq"),
                                   _dev(w_scale, torch.float32, (N,), "w_scale"), _stream_ptr(stream))
    _check(st, "jq_pack_weight_int4")
    return wq, w_scale


def jq_w4a4_linear(x, wq, w_scale, bias=None, y=None, workspace=None, stream=None):
    """y = W4A4 linear of x (bf16 [M,K]) with a packed weight; returns bf16 [M,N]."""
    torch = _torch()
    M, K = x.shape
    N = wq.shape[0]
    if y is None:
        y = torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    need = jq_w4a4_workspace_bytes(M, K)
    if workspace is None:
        workspace = torch.empty((need,), dtype=torch.uint8, device=x.device)
    bptr = ctypes.c_void_p(None) if bias is None else _dev(bias, torch.bfloat16, (N,), "bias")
    st = lib().jq_w4a4_linear(_dev(x, torch.bfloat16, None, "x"), M, K,
                              _dev(wq, torch.uint8, (N, K // 2), "wq"),
                              _dev(w_scale, torch.float32, (N,), "w_scale"), N, bptr,
                              _dev(y, torch.bfloat16, (M, N), "y"),
                              _dev(workspace, torch.uint8, None, "workspace"),
                              workspace.numel(), _stream_ptr(stream))
    _check(st, "jq_w4a4_linear")
    return y


def jq_w4a4_gemm(q, scale, wq, w_scale, bias=None, y=None, stream=None):
    """GEMM + epilogue on pre-quantised activations; returns bf16 [M,N]."""
    torch = _torch()
    M, Kh = q.shape
    K = 2 * Kh
    N = wq.shape[0]
    if y is None:
        y = torch.empty((M, N), dtype=torch.bfloat16, device=q.device)
    bptr = ctypes.c_void_p(None) if bias is None else _dev(bias, torch.bfloat16, (N,), "bias")
    st = lib().jq_w4a4_gemm(_dev(q, torch.uint8, (M, Kh), "q"), _dev(scale, torch.float32, (M,), "scale"),
                            M, K, _dev(wq, torch.uint8, (N, Kh), "wq"),
                            _dev(w_scale, torch.float32, (N,), "w_scale"), N, bptr,
                            _dev(y, torch.bfloat16, (M, N), "y"), _stream_ptr(stream))
    _check(st, "jq_w4a4_gemm")
    return y


def jq_w4a4_gemm_i32(q, wq, acc=None, stream=None):
    """Exact accumulators int32 [M,N] of the packed codes."""
    torch = _torch()
    M, Kh = q.shape
    N = wq.shape[0]
    if acc is None:
        acc = torch.empty((M, N), dtype=torch.int32, device=q.device)
    st = lib().jq_w4a4_gemm_i32(_dev(q, torch.uint8, (M, Kh), "q"), M, 2 * Kh,
                                _dev(wq, torch.uint8, (N, Kh), "wq"), N,
                                _dev(acc, torch.int32, (M, N), "acc"), _stream_ptr(stream))
    _check(st, "jq_w4a4_gemm_i32")
    return acc


# ---------------------------------------------------------------------------
# W1.58A4: ternary weights [N, K/4], same activation path
# ---------------------------------------------------------------------------


def jq_pack_weight_ternary(w, wt=None, w_scale=None, stream=None):
    """w bf16 [N,K] -> (wt uint8 [N,K/4] packed ternary codes, w_scale fp32 [N])."""
    torch = _torch()
    N, K = w.shape
    if wt is None:
        wt = torch.empty((N, K // 4), dtype=torch.uint8, device=w.device)
    if w_scale is None:
        w_scale = torch.empty((N,), dtype=torch.float32, device=w.device)
    st = lib().jq_pack_weight_ternary(_dev(w, torch.bfloat16, None, "w"), N, K,
                                      _dev(wt, torch.uint8, (N, K // 4), "wt"),
                                      _dev(w_scale, torch.float32, (N,), "w_scale"), _stream_ptr(stream))
    _check(st, "jq_pack_weight_ternary")
    return wt, w_scale


def jq_w158a4_linear(x, wt, w_scale, bias=None, y=None, workspace=None, stream=None):
    """y = W1.58A4 linear of x (bf16 [M,K]) with a packed ternary weight; returns bf16 [M,N]."""
    torch = _torch()
    M, K = x.shape
    N = wt.shape[0]
    if y is None:
        y = torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    need = jq_w4a4_workspace_bytes(M, K)
    if workspace is None:
        workspace = torch.empty((need,), dtype=torch.uint8, device=x.device)
    bptr = ctypes.c_void_p(None) if bias is None else _dev(bias, torch.bfloat16, (N,), "bias")
    st = lib().jq_w158a4_linear(_dev(x, torch.bfloat16, None, "x"), M, K,
                                _dev(wt, torch.uint8, (N, K // 4), "wt"),
                                _dev(w_scale, torch.float32, (N,), "w_scale"), N, bptr,
                                _dev(y, torch.bfloat16, (M, N), "y"),
                                _dev(workspace, torch.uint8, None, "workspace"),
                                workspace.numel(), _stream_ptr(stream))
    _check(st, "jq_w158a4_linear")
    return y


def jq_w158a4_gemm(q, scale, wt, w_scale, bias=None, y=None, stream=None):
    """GEMM + epilogue of pre-quantised activations with ternary weights; returns bf16 [M,N]."""
    torch = _torch()
    M, Kh = q.shape
    K = 2 * Kh
    N = wt.shape[0]
    if y is None:
        y = torch.empty((M, N), dtype=torch.bfloat16, device=q.device)
    bptr = ctypes.c_void_p(None) if bias is None else _dev(bias, torch.bfloat16, (N,), "bias")
    st = lib().jq_w158a4_gemm(_dev(q, torch.uint8, (M, Kh), "q"), _dev(scale, torch.float32, (M,), "scale"),
                              M, K, _dev(wt, torch.uint8, (N, K // 4), "wt"),
                              _dev(w_scale, torch.float32, (N,), "w_scale"), N, bptr,
                              _dev(y, torch.bfloat16, (M, N), "y"), _stream_ptr(stream))
    _check(st, "jq_w158a4_gemm")
    return y


def jq_w158a4_gemm_i32(q, wt, acc=None, stream=None):
    """Exact accumulators int32 [M,N] of int4 activation codes times ternary weight codes."""
    torch = _torch()
    M, Kh = q.shape
    K = 2 * Kh
    N = wt.shape[0]
    if acc is None:
        acc = torch.empty((M, N), dtype=torch.int32, device=q.device)
    st = lib().jq_w158a4_gemm_i32(_dev(q, torch.uint8, (M, Kh), "q"), M, K,
                                  _dev(wt, torch.uint8, (N, K // 4), "wt"), N,
                                  _dev(acc, torch.int32, (M, N), "acc"), _stream_ptr(stream))
    _check(st, "jq_w158a4_gemm_i32")
    return acc


# ---------------------------------------------------------------------------
# group-wise W4A4: scales [rows, K/G], G = 64 or 128
# ---------------------------------------------------------------------------


def jq_w4a4g_workspace_bytes(M, K, G):
    return int(lib().jq_w4a4g_workspace_bytes(int(M), int(K), int(G)))


def _quantize_group(fn, name, x, G, q, scale, stream):
    torch = _torch()
    R, K = x.shape
    if q is None:
        q = torch.empty((R, K // 2), dtype=torch.uint8, device=x.device)
    if scale is None:
        scale = torch.empty((R, K // G), dtype=torch.float32, device=x.device)
    st = fn(_dev(x, torch.bfloat16, None, "x"), R, K, G, _dev(q, torch.uint8, (R, K // 2), "q"),
            _dev(scale, torch.float32, (R, K // G), "scale"), _stream_ptr(stream))
    _check(st, name)
    return q, scale


def jq_quantize_act_group(x, G, q=None, scale=None, stream=None):
    """x bf16 [M,K] -> (q uint8 [M,K/2], scales fp32 [M,K/G])."""
    return _quantize_group(lib().jq_quantize_act_group, "jq_quantize_act_group", x, G, q, scale, stream)


def jq_pack_weight_int4_group(w, G, wq=None, w_scale=None, stream=None):
    """w bf16 [N,K] -> (wq uint8 [N,K/2], w_scales fp32 [N,K/G])."""
    return _quantize_group(lib().jq_pack_weight_int4_group, "jq_pack_weight_int4_group", w, G, wq, w_scale, stream)


def jq_w4a4g_linear(x, wq, w_scale, G, bias=None, y=None, workspace=None, stream=None):
    """y = group-wise W4A4 linear of x (bf16 [M,K]); returns bf16 [M,N]."""
    torch = _torch()
    M, K = x.shape
    N = wq.shape[0]
    if y is None:
        y = torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    if workspace is None:
        workspace = torch.empty((jq_w4a4g_workspace_bytes(M, K, G),), dtype=torch.uint8, device=x.device)
    bptr = ctypes.c_void_p(None) if bias is None else _dev(bias, torch.bfloat16, (N,), "bias")
    st = lib().jq_w4a4g_linear(_dev(x, torch.bfloat16, None, "x"), M, K, G,
                               _dev(wq, torch.uint8, (N, K // 2), "wq"),
                               _dev(w_scale, torch.float32, (N, K // G), "w_scale"), N, bptr,
                               _dev(y, torch.bfloat16, (M, N), "y"),
                               _dev(workspace, torch.uint8, None, "workspace"), workspace.numel(),
                               _stream_ptr(stream))
    _check(st, "jq_w4a4g_linear")
    return y


def jq_w4a4g_gemm(q, scale, wq, w_scale, G, bias=None, y=None, stream=None):
    """Group GEMM + epilogue on pre-quantised activations; returns bf16 [M,N]."""
    torch = _torch()
    M, Kh = q.shape
    K = 2 * Kh
    N = wq.shape[0]
    if y is None:
        y = torch.empty((M, N), dtype=torch.bfloat16, device=q.device)
    bptr = ctypes.c_void_p(None) if bias is None else _dev(bias, torch.bfloat16, (N,), "bias")
    st = lib().jq_w4a4g_gemm(_dev(q, torch.uint8, (M, Kh), "q"), _dev(scale, torch.float32, (M, K // G), "scale"),
                             M, K, G, _dev(wq, torch.uint8, (N, Kh), "wq"),
                             _dev(w_scale, torch.float32, (N, K // G), "w_scale"), N, bptr,
                             _dev(y, torch.bfloat16, (M, N), "y"), _stream_ptr(stream))
    _check(st, "jq_w4a4g_gemm")
    return y


def jq_w4a4g_gemm_f32(q, scale, wq, w_scale, G, out=None, stream=None):
    """The fp32 group sum S [M,N] (before bias and bf16 rounding)."""
    torch = _torch()
    M, Kh = q.shape
    K = 2 * Kh
    N = wq.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=q.device)
    st = lib().jq_w4a4g_gemm_f32(_dev(q, torch.uint8, (M, Kh), "q"),
                                 _dev(scale, torch.float32, (M, K // G), "scale"), M, K, G,
                                 _dev(wq, torch.uint8, (N, Kh), "wq"),
                                 _dev(w_scale, torch.float32, (N, K // G), "w_scale"), N,
                                 _dev(out, torch.float32, (M, N), "out"), _stream_ptr(stream))
    _check(st, "jq_w4a4g_gemm_f32")
    return out


# ---------------------------------------------------------------------------
# BF6 engine: the same layer on the 6-bit matrix cores (operands in the BF6
# layout of include/jq.h, held as flat uint8 tensors)
# ---------------------------------------------------------------------------


def jq_f6_operand_bytes(rows, K):
    return int(lib().jq_f6_operand_bytes(int(rows), int(K)))


def jq_w4a4_f6_workspace_bytes(M, K):
    return int(lib().jq_w4a4_f6_workspace_bytes(int(M), int(K)))


def jq_gemm_plan(M, N, K, cus):
    """Tile rows (128 or 112) the int8 engine's GEMM takes for an M x K by K x N product on `cus` CUs (host only)."""
    t = ctypes.c_int(0)
    st = lib().jq_gemm_plan(int(M), int(N), int(K), int(cus), ctypes.byref(t))
    _check(st, "jq_gemm_plan")
    return t.value


def jq_f6_gemm_plan(M, N, K, cus):
    """(waves, tile_rows) the BF6 GEMM takes for an M x K by K x N product on `cus` CUs (host only)."""
    w, t = ctypes.c_int(0), ctypes.c_int(0)
    st = lib().jq_f6_gemm_plan(int(M), int(N), int(K), int(cus), ctypes.byref(w), ctypes.byref(t))
    _check(st, "jq_f6_gemm_plan")
    return w.value, t.value


def jq_quantize_act_f6(x, xf6=None, scale=None, stream=None):
    """x bf16 [M,K] -> (BF6 activation operand uint8 [jq_f6_operand_bytes(M,K)], scale fp32 [M])."""
    torch = _torch()
    M, K = x.shape
    nb = jq_f6_operand_bytes(M, K)
    if xf6 is None:
        xf6 = torch.empty((nb,), dtype=torch.uint8, device=x.device)
    if scale is None:
        scale = torch.empty((M,), dtype=torch.float32, device=x.device)
    st = lib().jq_quantize_act_f6(_dev(x, torch.bfloat16, None, "x"), M, K, _dev(xf6, torch.uint8, (nb,), "xf6"),
                                  _dev(scale, torch.float32, (M,), "scale"), _stream_ptr(stream))
    _check(st, "jq_quantize_act_f6")
    return xf6, scale


def _int4_to_f6(name, q, out, stream, codes_per_byte=2):
    torch = _torch()
    rows, Kb = q.shape
    K = codes_per_byte * Kb
    nb = jq_f6_operand_bytes(rows, K)
    if out is None:
        out = torch.empty((nb,), dtype=torch.uint8, device=q.device)
    st = getattr(lib(), name)(_dev(q, torch.uint8, (rows, Kb), "q"), rows, K,
                              _dev(out, torch.uint8, (nb,), "out"), _stream_ptr(stream))
    _check(st, name)
    return out


def jq_int4_to_f6(q, out=None, stream=None):
    """Packed int4 codes uint8 [rows,K/2] -> BF6 operand, activation layout, uint8 [jq_f6_operand_bytes(rows,K)]."""
    return _int4_to_f6("jq_int4_to_f6", q, out, stream)


def jq_int4_to_f6_weight(q, out=None, stream=None):
    """Packed int4 codes uint8 [rows,K/2] -> BF6 operand, weight layout, uint8 [jq_f6_operand_bytes(rows,K)]."""
    return _int4_to_f6("jq_int4_to_f6_weight", q, out, stream)


def jq_ternary_to_f6_weight(wt, out=None, stream=None):
    """Packed ternary codes uint8 [rows,K/4] -> BF6 operand, weight layout, uint8 [jq_f6_operand_bytes(rows,K)].

    With the ternary scales as w_scale, jq_w4a4_f6_linear then computes the W1.58A4 layer."""
    return _int4_to_f6("jq_ternary_to_f6_weight", wt, out, stream, codes_per_byte=4)


def jq_w4a4_f6_linear(x, wf6, w_scale, bias=None, y=None, workspace=None, stream=None):
    """y = W4A4 linear of x (bf16 [M,K]) on the BF6 engine; returns bf16 [M,N]."""
    torch = _torch()
    M, K = x.shape
    N = w_scale.shape[0]
    if y is None:
        y = torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    if workspace is None:
        workspace = torch.empty((jq_w4a4_f6_workspace_bytes(M, K),), dtype=torch.uint8, device=x.device)
    bptr = ctypes.c_void_p(None) if bias is None else _dev(bias, torch.bfloat16, (N,), "bias")
    st = lib().jq_w4a4_f6_linear(_dev(x, torch.bfloat16, None, "x"), M, K,
                                 _dev(wf6, torch.uint8, (jq_f6_operand_bytes(N, K),), "wf6"),
                                 _dev(w_scale, torch.float32, (N,), "w_scale"), N, bptr,
                                 _dev(y, torch.bfloat16, (M, N), "y"),
                                 _dev(workspace, torch.uint8, None, "workspace"), workspace.numel(),
                                 _stream_ptr(stream))
    _check(st, "jq_w4a4_f6_linear")
    return y


JQ_QUANT_BATCH_MAX = 8


def jq_quantize_act_f6_batch(xs, xf6s=None, scales=None, stream=None):
    """Per-token BF6 quantisation of several independent bf16 [M_i, K_i] inputs in
    one call; returns (list of BF6 operands, list of scales)."""
    torch = _torch()
    n = len(xs)
    if xf6s is None:
        xf6s = [torch.empty((jq_f6_operand_bytes(*x.shape),), dtype=torch.uint8, device=x.device) for x in xs]
    if scales is None:
        scales = [torch.empty((x.shape[0],), dtype=torch.float32, device=x.device) for x in xs]
    if not (len(xf6s) == len(scales) == n):
        raise ValueError("xs, xf6s and scales must have the same length")
    ptrs = lambda vals: (ctypes.c_void_p * max(n, 1))(*[v.value for v in vals])
    xp = ptrs([_dev(x, torch.bfloat16, None, f"xs[{i}]") for i, x in enumerate(xs)])
    qp = ptrs([_dev(q, torch.uint8, (jq_f6_operand_bytes(*x.shape),), f"xf6s[{i}]")
               for i, (x, q) in enumerate(zip(xs, xf6s))])
    sp = ptrs([_dev(s, torch.float32, (x.shape[0],), f"scales[{i}]") for i, (x, s) in enumerate(zip(xs, scales))])
    Ms = (ctypes.c_int64 * max(n, 1))(*[x.shape[0] for x in xs])
    Ks = (ctypes.c_int64 * max(n, 1))(*[x.shape[1] for x in xs])
    st = lib().jq_quantize_act_f6_batch(n, xp, Ms, Ks, qp, sp, _stream_ptr(stream))
    _check(st, "jq_quantize_act_f6_batch")
    return xf6s, scales


# The library-held scratch of jq_w4a4_f6_linear_noalloc, per device (include/jq.h).
JQ_NOALLOC_SCRATCH_BYTES = 96 << 20


def jq_w4a4_f6_linear_noalloc(x, wf6, w_scale, bias=None, y=None, stream=None):
    """jq_w4a4_f6_linear with its workspace in the library's own device scratch
    (allocates nothing itself; calls that overlap on one device race); returns bf16 [M,N]."""
    torch = _torch()
    M, K = x.shape
    N = w_scale.shape[0]
    if y is None:
        y = torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    bptr = ctypes.c_void_p(None) if bias is None else _dev(bias, torch.bfloat16, (N,), "bias")
    st = lib().jq_w4a4_f6_linear_noalloc(_dev(x, torch.bfloat16, None, "x"), M, K,
                                         _dev(wf6, torch.uint8, (jq_f6_operand_bytes(N, K),), "wf6"),
                                         _dev(w_scale, torch.float32, (N,), "w_scale"), N, bptr,
                                         _dev(y, torch.bfloat16, (M, N), "y"), _stream_ptr(stream))
    _check(st, "jq_w4a4_f6_linear_noalloc")
    return y


def jq_w4a4_f6_gemm(xf6, scale, K, wf6, w_scale, bias=None, y=None, stream=None):
    """GEMM + epilogue of the BF6 engine on a quantised activation operand; returns bf16 [M,N]."""
    torch = _torch()
    M, N = scale.shape[0], w_scale.shape[0]
    if y is None:
        y = torch.empty((M, N), dtype=torch.bfloat16, device=xf6.device)
    bptr = ctypes.c_void_p(None) if bias is None else _dev(bias, torch.bfloat16, (N,), "bias")
    st = lib().jq_w4a4_f6_gemm(_dev(xf6, torch.uint8, (jq_f6_operand_bytes(M, K),), "xf6"),
                               _dev(scale, torch.float32, (M,), "scale"), M, K,
                               _dev(wf6, torch.uint8, (jq_f6_operand_bytes(N, K),), "wf6"),
                               _dev(w_scale, torch.float32, (N,), "w_scale"), N, bptr,
                               _dev(y, torch.bfloat16, (M, N), "y"), _stream_ptr(stream))
    _check(st, "jq_w4a4_f6_gemm")
    return y


def jq_w4a4_f6_gemm_i32(xf6, M, K, wf6, N, acc=None, stream=None):
    """Exact accumulators int32 [M,N] of two BF6 operands."""
    torch = _torch()
    if acc is None:
        acc = torch.empty((M, N), dtype=torch.int32, device=xf6.device)
    st = lib().jq_w4a4_f6_gemm_i32(_dev(xf6, torch.uint8, (jq_f6_operand_bytes(M, K),), "xf6"), M, K,
                                   _dev(wf6, torch.uint8, (jq_f6_operand_bytes(N, K),), "wf6"), N,
                                   _dev(acc, torch.int32, (M, N), "acc"), _stream_ptr(stream))
    _check(st, "jq_w4a4_f6_gemm_i32")
    return acc


# ---------------------------------------------------------------------------
# host <-> device helpers for bf16 bit patterns (data movement only)
# ---------------------------------------------------------------------------


def bf16_tensor(bits, device="cuda"):
    """numpy uint16 bf16 bit patterns -> torch.bfloat16 tensor on `device`."""
    import numpy as np

    torch = _torch()
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    return t.to(device)


def bf16_bits(t):
    """torch.bfloat16 tensor -> numpy uint16 bit patterns (on the host)."""
    import numpy as np

    torch = _torch()
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


# ---------------------------------------------------------------------------
# group-wise W4A4 on the BF6 engine: BF6 operands, scales [rows, K/G]
# ---------------------------------------------------------------------------


def jq_w4a4g_f6_workspace_bytes(M, K, G):
    return int(lib().jq_w4a4g_f6_workspace_bytes(int(M), int(K), int(G)))


def jq_quantize_act_group_f6(x, G, xf6=None, scale=None, stream=None):
    """x bf16 [M,K] -> (BF6 activation operand uint8 [jq_f6_operand_bytes(M,K)], scales fp32 [M,K/G])."""
    torch = _torch()
    M, K = x.shape
    nb = jq_f6_operand_bytes(M, K)
    if xf6 is None:
        xf6 = torch.empty((nb,), dtype=torch.uint8, device=x.device)
    if scale is None:
        scale = torch.empty((M, K // G), dtype=torch.float32, device=x.device)
    st = lib().jq_quantize_act_group_f6(_dev(x, torch.bfloat16, None, "x"), M, K, G,
                                        _dev(xf6, torch.uint8, (nb,), "xf6"),
                                        _dev(scale, torch.float32, (M, K // G), "scale"), _stream_ptr(stream))
    _check(st, "jq_quantize_act_group_f6")
    return xf6, scale


def jq_w4a4g_f6_linear(x, wf6, w_scale, G, bias=None, y=None, workspace=None, stream=None):
    """y = group-wise W4A4 linear of x (bf16 [M,K]) on the BF6 engine; wf6 from
    jq_int4_to_f6_weight of jq_pack_weight_int4_group's codes, w_scale its scales [N,K/G]."""
    torch = _torch()
    M, K = x.shape
    N = w_scale.shape[0]
    if y is None:
        y = torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    if workspace is None:
        workspace = torch.empty((jq_w4a4g_f6_workspace_bytes(M, K, G),), dtype=torch.uint8, device=x.device)
    bptr = ctypes.c_void_p(None) if bias is None else _dev(bias, torch.bfloat16, (N,), "bias")
    st = lib().jq_w4a4g_f6_linear(_dev(x, torch.bfloat16, None, "x"), M, K, G,
                                  _dev(wf6, torch.uint8, (jq_f6_operand_bytes(N, K),), "wf6"),
                                  _dev(w_scale, torch.float32, (N, K // G), "w_scale"), N, bptr,
                                  _dev(y, torch.bfloat16, (M, N), "y"),
                                  _dev(workspace, torch.uint8, None, "workspace"), workspace.numel(),
                                  _stream_ptr(stream))
    _check(st, "jq_w4a4g_f6_linear")
    return y


def jq_w4a4g_f6_gemm(xf6, scale, wf6, w_scale, G, bias=None, y=None, stream=None):
    """Group GEMM + epilogue on the BF6 engine (scale [M,K/G], w_scale [N,K/G]); returns bf16 [M,N]."""
    torch = _torch()
    M, KG = scale.shape
    N = w_scale.shape[0]
    K = KG * G
    if y is None:
        y = torch.empty((M, N), dtype=torch.bfloat16, device=xf6.device)
    bptr = ctypes.c_void_p(None) if bias is None else _dev(bias, torch.bfloat16, (N,), "bias")
    st = lib().jq_w4a4g_f6_gemm(_dev(xf6, torch.uint8, (jq_f6_operand_bytes(M, K),), "xf6"),
                                _dev(scale, torch.float32, (M, KG), "scale"), M, K, G,
                                _dev(wf6, torch.uint8, (jq_f6_operand_bytes(N, K),), "wf6"),
                                _dev(w_scale, torch.float32, (N, KG), "w_scale"), N, bptr,
                                _dev(y, torch.bfloat16, (M, N), "y"), _stream_ptr(stream))
    _check(st, "jq_w4a4g_f6_gemm")
    return y


def jq_w4a4g_f6_gemm_f32(xf6, scale, wf6, w_scale, G, out=None, stream=None):
    """The fp32 group sum S [M,N] of the BF6 group GEMM (before bias and bf16 rounding)."""
    torch = _torch()
    M, KG = scale.shape
    N = w_scale.shape[0]
    K = KG * G
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=xf6.device)
    st = lib().jq_w4a4g_f6_gemm_f32(_dev(xf6, torch.uint8, (jq_f6_operand_bytes(M, K),), "xf6"),
                                    _dev(scale, torch.float32, (M, KG), "scale"), M, K, G,
                                    _dev(wf6, torch.uint8, (jq_f6_operand_bytes(N, K),), "wf6"),
                                    _dev(w_scale, torch.float32, (N, KG), "w_scale"), N,
                                    _dev(out, torch.float32, (M, N), "out"), _stream_ptr(stream))
    _check(st, "jq_w4a4g_f6_gemm_f32")
    return out
