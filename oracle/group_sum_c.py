"""Compiled group-wise steps 6-7 for whole full-size checks (test infrastructure only).

The numpy oracle (w4a4_group.py) computes the group-wise fp32 sums through an
[M, N, K/G] array of exact accumulators; at the workload sizes that is tens of
GB and minutes per layer.  group_sum.c computes the same sums output by
output with a plain loop nest: per group the exact integer dot product of
the two code slices, times the activation scale, times the weight scale
(each rounded to fp32), added to the running fp32 sum in group order from +0.
The CPU tests require it to equal the numpy oracle bit for bit, on random and
extreme operands, so that the GPU tests may use it in its place at full size.

The caller here only splits the output into rectangles and runs them on a
pool of threads (ctypes releases the GIL during each call); every output is
computed by one call, whole.  Only the tests may import this module.
"""

import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .w4a4 import unpack_int4

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "group_sum.c")
LIB_PATH = os.path.join(_HERE, "_group_sum.so")
CFLAGS = ["-O3", "-ffp-contract=off", "-fno-fast-math", "-fno-strict-aliasing", "-shared", "-fPIC"]

_lib = None


def build():
    """Compile group_sum.c into oracle/_group_sum.so with gcc; returns the path."""
    tmp = LIB_PATH + ".tmp"
    subprocess.run(["gcc", *CFLAGS, SOURCE, "-o", tmp], check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def load(path):
    """The rectangle function of a compiled group_sum.c at path."""
    f = ctypes.CDLL(path).oracle_group_sum_rect
    i64, p = ctypes.c_int64, ctypes.c_void_p
    f.argtypes = [p, p, p, p, i64, i64, i64, i64, i64, i64, i64, p]
    f.restype = None
    return f


def lib():
    """The rectangle function of oracle/_group_sum.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built (oracle.group_sum_c.build())")
        _lib = load(LIB_PATH)
    return _lib


def _threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def group_sum_codes(qx, s_x, qw, s_w, G, tile=(32, 64), threads=None, fn=None):
    """S [M, N] fp32 from int8 codes qx [M, K], qw [N, K] and fp32 group scales
    (fn: another build's rectangle function, for the tests that check the pins)."""
    qx = np.ascontiguousarray(qx, dtype=np.int8)
    qw = np.ascontiguousarray(qw, dtype=np.int8)
    s_x = np.ascontiguousarray(s_x, dtype=np.float32)
    s_w = np.ascontiguousarray(s_w, dtype=np.float32)
    M, K = qx.shape
    N = qw.shape[0]
    assert qw.shape[1] == K and G > 0 and K % G == 0 and G <= 1 << 18
    assert s_x.shape == (M, K // G) and s_w.shape == (N, K // G)
    S = np.empty((M, N), dtype=np.float32)
    if M == 0 or N == 0:
        return S
    f = fn or lib()
    tm, tn = tile
    ptrs = [a.ctypes.data for a in (qx, s_x, qw, s_w)]

    def rows(m0):
        m1 = min(M, m0 + tm)
        for n0 in range(0, N, tn):
            f(*ptrs, N, K, G, m0, m1, n0, min(N, n0 + tn), S.ctypes.data)

    with ThreadPoolExecutor(threads or _threads()) as ex:
        list(ex.map(rows, range(0, M, tm)))
    return S


def w4a4g_gemm_f32(qx_packed, s_x, qw_packed, s_w, G, threads=None):
    """Same result as the numpy oracle's w4a4g_gemm_f32, from packed codes."""
    return group_sum_codes(unpack_int4(qx_packed), s_x, unpack_int4(qw_packed), s_w, G, threads=threads)
