"""The paper's ISC on the host CPU (Sec. "Sparse Convolution", steps 1-3),
and the host im2col of Fig. 3: for timing the CPU speedup trend of Tab. 2
beside a BLAS GEMM on the same host.  ctypes over libisc_host.so (built by
paper_1704_07724_amd.build); argument marshalling only.  Not used by the GPU
path."""
from __future__ import annotations

import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libisc_host.so")
_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("%s is missing: run python -m paper_1704_07724_amd.build" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        fp = ctypes.POINTER(ctypes.c_float)
        L.isc_host_repack.argtypes = [fp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, fp]
        L.isc_host_repack.restype = None
        L.isc_host_conv2d.argtypes = [fp, fp, fp] + [ctypes.c_int] * 10
        L.isc_host_conv2d.restype = ctypes.c_int
        L.isc_host_im2col.argtypes = [fp] + [ctypes.c_int] * 7 + [fp]
        L.isc_host_im2col.restype = None
        _lib = L
    return _lib


def _f32(a) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def out_shape(H, W, R, S, T, P):
    return (H + 2 * P - R) // T + 1, (W + 2 * P - S) // T + 1


def repack(w) -> np.ndarray:
    """K x C x R x S -> [C][R][S][K] (ISC step 2's K-contiguous layout)."""
    w = _f32(w)
    K, C, R, S = w.shape
    wt = np.empty((C, R, S, K), dtype=np.float32)
    lib().isc_host_repack(_ptr(w), K, C, R, S, _ptr(wt))
    return wt


def conv2d(x, wt, stride=1, pad=0, threads=1, out=None) -> np.ndarray:
    """y = conv(x, w) by ISC on the host; wt from repack()."""
    x, wt = _f32(x), _f32(wt)
    N, C, H, W = x.shape
    C2, R, S, K = wt.shape
    if C2 != C:
        raise ValueError("filter has %d input maps, input %d" % (C2, C))
    Ho, Wo = out_shape(H, W, R, S, stride, pad)
    if Ho < 1 or Wo < 1 or stride < 1 or pad < 0:
        raise ValueError("bad convolution shape")
    y = out if out is not None else np.empty((N, K, Ho, Wo), dtype=np.float32)
    if y.shape != (N, K, Ho, Wo) or y.dtype != np.float32 or not y.flags.c_contiguous:
        raise ValueError("out must be a C-contiguous float32 array of shape %s" % ((N, K, Ho, Wo),))
    if lib().isc_host_conv2d(_ptr(x), _ptr(wt), _ptr(y), N, C, H, W, K, R, S, stride, pad, int(threads)) != 0:
        raise MemoryError("isc_host_conv2d: no scratch memory")
    return y


def im2col(x1, R, S, stride=1, pad=0) -> np.ndarray:
    """Fig. 3's (C*R*S) x (Ho*Wo) input matrix of one image x1 [C][H][W]."""
    x1 = _f32(x1)
    C, H, W = x1.shape
    Ho, Wo = out_shape(H, W, R, S, stride, pad)
    col = np.empty((C * R * S, Ho * Wo), dtype=np.float32)
    lib().isc_host_im2col(_ptr(x1), C, H, W, R, S, stride, pad, _ptr(col))
    return col
