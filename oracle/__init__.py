"""CPU reference ("oracle") for the sparse-input convolution -- TEST INFRASTRUCTURE.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports, links or calls it, and the two share no
code: the arithmetic lives in ``isc_oracle.c`` (plain C, fp64 accumulation,
written from the paper), this module only marshals numpy arrays.

What each function follows (Shi & Chu, arXiv 1704.07724):
  conv2d_f64 / conv2d_f64_at   Eq. 1 (Sec. "Sparsity of ReLUs") with batch,
                               stride T and zero padding P added
  out_size                     output size of Sec. "Sparsity of ReLUs", read
                               as floor((H + 2P - R)/T) + 1
  compact                      ISC step 1 (Sec. "Sparse Convolution"):
                               row-major nonzero list per (n, c) plane
  nz_macs                      exact count of the multiply-adds ISC performs
                               (the rho * Ho*Wo*R*S*K*C estimate of
                               Sec. "Sparse Convolution", border-exact)
  im2col                       the unrolled input matrix M_I of the
                               matrix-multiplication formulation (Fig. 3)
  relu_conv2d_f64              Eq. 1 followed by the rectifier of Eq. 2
                               (Sec. "Sparsity of ReLUs"), with the nonzero
                               count of the rectified output
  conv2d_dw_f64                the weight gradient of Eq. 1 (training, whose
                               rectified inputs the paper measures in Sec.
                               "Sparsity of ReLUs")

Pins (tests/test_oracle_pins.py) tie each function to something other than
itself: brute-force loops, closed forms, numpy / torch library routines,
invariants.  No function here is "parity unpinned".
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "isc_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True, src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile isc_oracle.c into liboracle.so next to it (gcc, OpenMP)."""
    if force or not os.path.exists(out):
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c99",
             "-Wall", "-Wextra", "-o", tmp, src])
        os.replace(tmp, out)
    return out


def load_library(path: str):
    """ctypes handle with the oracle's signatures declared."""
    lib = ctypes.CDLL(path)
    i32, i64 = ctypes.c_int, ctypes.c_int64
    vp = ctypes.c_void_p
    lib.oracle_out_size.argtypes = [i32, i32, i32, i32]
    lib.oracle_out_size.restype = i32
    lib.oracle_conv2d_f64.argtypes = [vp, vp] + [i32] * 9 + [vp]
    lib.oracle_conv2d_f64.restype = None
    lib.oracle_conv2d_f64_at.argtypes = [vp, vp] + [i32] * 9 + [vp, i64, vp]
    lib.oracle_conv2d_f64_at.restype = None
    lib.oracle_compact.argtypes = [vp, i32, i32, i32, i32, vp, vp, vp, vp]
    lib.oracle_compact.restype = i64
    lib.oracle_nz_macs.argtypes = [vp] + [i32] * 9
    lib.oracle_nz_macs.restype = i64
    lib.oracle_im2col.argtypes = [vp] + [i32] * 8 + [i64, vp]
    lib.oracle_im2col.restype = None
    lib.oracle_conv2d_dw_f64.argtypes = [vp, vp] + [i32] * 9 + [vp]
    lib.oracle_conv2d_dw_f64.restype = None
    lib.oracle_rectify_f64.argtypes = [vp, i64]
    lib.oracle_rectify_f64.restype = i64
    lib.oracle_threads.argtypes = []
    lib.oracle_threads.restype = i32
    lib.oracle_set_threads.argtypes = [i32]
    lib.oracle_set_threads.restype = None
    return lib


def _load():
    global _lib
    if _lib is None:
        # ISC_ORACLE_LIB names another build of the oracle; the mutation test
        # uses it to run the pins against deliberately broken copies
        alt = os.environ.get("ISC_ORACLE_LIB")
        if alt:
            _lib = load_library(alt)
        else:
            if not os.path.exists(_LIB_PATH):
                build(force=True)
            _lib = load_library(_LIB_PATH)
    return _lib


def _f32(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.float32:
        raise TypeError("oracle expects float32 arrays, got %s" % a.dtype)
    return a


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_load().oracle_threads())


def set_threads(n: int) -> None:
    """Thread count of the oracle's parallel loops from now on (timing only)."""
    _load().oracle_set_threads(int(n))


def out_size(n_in: int, k: int, pad: int, stride: int) -> int:
    return int(_load().oracle_out_size(n_in, k, pad, stride))


def out_shape(x_shape, w_shape, stride: int, pad: int):
    N, C, H, W = x_shape
    K, C2, R, S = w_shape
    assert C == C2
    return (N, K, out_size(H, R, pad, stride), out_size(W, S, pad, stride))


def conv2d_f64(x, w, stride: int = 1, pad: int = 0) -> np.ndarray:
    """Direct convolution of Eq. 1 (batch, stride, zero padding), fp64 output."""
    x, w = _f32(x), _f32(w)
    N, C, H, W = x.shape
    K, C2, R, S = w.shape
    if C != C2:
        raise ValueError("channel mismatch")
    shp = out_shape(x.shape, w.shape, stride, pad)
    out = np.empty(shp, dtype=np.float64)
    if out.size:
        _load().oracle_conv2d_f64(_ptr(x), _ptr(w), N, C, H, W, K, R, S,
                                  stride, pad, _ptr(out))
    return out


def conv2d_f64_at(x, w, stride: int, pad: int, flat_idx) -> np.ndarray:
    """Eq. 1 evaluated at the given flat NCHW output indices only."""
    x, w = _f32(x), _f32(w)
    N, C, H, W = x.shape
    K, _, R, S = w.shape
    idx = np.ascontiguousarray(flat_idx, dtype=np.int64)
    out = np.empty(idx.shape, dtype=np.float64)
    if idx.size:
        _load().oracle_conv2d_f64_at(_ptr(x), _ptr(w), N, C, H, W, K, R, S,
                                     stride, pad, _ptr(idx), idx.size, _ptr(out))
    return out


def relu_conv2d_f64(x, w, stride: int = 1, pad: int = 0):
    """Eq. 1 then the rectifier max(0, v) of Eq. 2, fp64; returns (y, nnz),
    nnz the number of nonzero entries of y (the next layer's nonzero count)."""
    y = conv2d_f64(x, w, stride, pad)
    nnz = int(_load().oracle_rectify_f64(_ptr(y), y.size)) if y.size else 0
    return y, nnz


def conv2d_dw_f64(x, dy, R: int, S: int, stride: int = 1, pad: int = 0) -> np.ndarray:
    """Weight gradient of Eq. 1: dw[k,c,r,s] = sum over n, i, j of
    dy[n,k,i,j] * X^[n, c, i*T + r - P, j*T + s - P], fp64 (K x C x R x S)."""
    x, dy = _f32(x), _f32(dy)
    N, C, H, W = x.shape
    Ho, Wo = out_size(H, R, pad, stride), out_size(W, S, pad, stride)
    if dy.shape[0] != N or dy.shape[2:] != (Ho, Wo):
        raise ValueError("dy must be N x K x Ho x Wo")
    K = dy.shape[1]
    dw = np.zeros((K, C, R, S), dtype=np.float64)
    if dw.size and Ho > 0 and Wo > 0:
        _load().oracle_conv2d_dw_f64(_ptr(x), _ptr(dy), N, C, H, W, K, R, S, stride, pad, _ptr(dw))
    return dw


def compact(x):
    """ISC step 1: per (n, c) plane, row-major nonzero list.

    Returns (row_ptr[N*C, H+1] int32, v[N*C, H*W] float32, ys, xs int32,
    total).  Slots past a plane's count are zero.
    """
    x = _f32(x)
    N, C, H, W = x.shape
    row_ptr = np.zeros((N * C, H + 1), dtype=np.int32)
    v = np.zeros((N * C, H * W), dtype=np.float32)
    ys = np.zeros((N * C, H * W), dtype=np.int32)
    xs = np.zeros((N * C, H * W), dtype=np.int32)
    total = _load().oracle_compact(_ptr(x), N, C, H, W, _ptr(row_ptr),
                                   _ptr(v), _ptr(ys), _ptr(xs))
    return row_ptr, v, ys, xs, int(total)


def nz_macs(x, K: int, R: int, S: int, stride: int, pad: int) -> int:
    """Exact multiply-add count of the zero-skipping convolution."""
    x = _f32(x)
    N, C, H, W = x.shape
    return int(_load().oracle_nz_macs(_ptr(x), N, C, H, W, K, R, S, stride, pad))


def im2col(x, R: int, S: int, stride: int, pad: int, ldc: int | None = None):
    """Unrolled input matrix M_I: rows (c, r, s), columns (n, i, j)."""
    x = _f32(x)
    N, C, H, W = x.shape
    Ho, Wo = out_size(H, R, pad, stride), out_size(W, S, pad, stride)
    ncols = N * Ho * Wo
    ldc = ncols if ldc is None else int(ldc)
    col = np.zeros((C * R * S, ldc), dtype=np.float32)
    if col.size:
        _load().oracle_im2col(_ptr(x), N, C, H, W, R, S, stride, pad, ldc, _ptr(col))
    return col


def sparsity(x) -> float:
    """Fraction of zero inputs (bit test with the sign cleared), the sparsity
    1 - rho of Sec. "Sparse Convolution" over the whole call."""
    x = _f32(x)
    if x.size == 0:
        return 0.0
    _, _, _, _, total = compact(x)
    return 1.0 - total / x.size
