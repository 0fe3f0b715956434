"""Python binding of libisc.so, the MI355X sparse-input convolution library.

Argument marshalling only: every step of the computation runs in the HIP
kernels behind the C ABI declared in include/isc.h; torch supplies device
memory and the current stream.  The binding refuses to work without the built
library (there is no fallback of any kind).

The functions carry the C names:
    isc_out_shape, isc_workspace_size, isc_conv2d (isc_conv2d_tuned when a
    tuning is given), isc_conv2d_noalloc, isc_decision, isc_read_decision,
    isc_census_size, isc_conv2d_relu, isc_census_read,
    isc_conv2d_dw_workspace_size, isc_conv2d_dw,
    isc_compact, isc_repacked_filter_size, isc_repack_filter,
    isc_sparse_conv, isc_sparse_conv_fused, isc_sparse_kernel, isc_sparse_plan,
    isc_crossover_sparsity,
    isc_im2col, isc_gemm_f32, isc_status_str, isc_version

Defaults a user may set in the environment (read here, by the binding, at
each call; the C library reads no environment): ISC_PATH = auto | sparse |
dense (the path when a call names none) and ISC_SPARSE_THRESHOLD (AUTO's
fixed sparsity threshold when a call names none; unset, AUTO uses the
library's per-shape crossover).

Stream safety: every temporary (workspace, contiguous copies, outputs) is
allocated on the stream the call is enqueued on, so torch's caching
allocator never hands it to another stream while the kernels still use it.
"""
from __future__ import annotations

import contextlib
import ctypes
import os

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libisc.so")

PATHS = {"auto": 0, "sparse": 1, "dense": 2}
PATH_NAMES = {v: k for k, v in PATHS.items()}

ISC_OK = 0
STATUS = {
    0: "ISC_OK", 1: "ISC_ERR_NULL", 2: "ISC_ERR_SHAPE", 3: "ISC_ERR_LIMIT",
    4: "ISC_ERR_WORKSPACE", 5: "ISC_ERR_ALIAS", 6: "ISC_ERR_PATH", 7: "ISC_ERR_DEVICE",
    8: "ISC_ERR_HIP", 9: "ISC_ERR_ALIGN", 10: "ISC_ERR_ARG",
}
EXPORTS = ("isc_out_shape", "isc_workspace_size", "isc_conv2d", "isc_conv2d_tuned", "isc_decision",
           "isc_read_decision", "isc_sparse_plan", "isc_conv2d_noalloc", "isc_crossover_sparsity",
           "isc_compact", "isc_repacked_filter_size", "isc_repack_filter", "isc_sparse_conv",
           "isc_im2col", "isc_gemm_f32", "isc_sparse_conv_fused", "isc_sparse_kernel",
           "isc_census_size", "isc_conv2d_relu", "isc_census_read",
           "isc_conv2d_dw_workspace_size", "isc_conv2d_dw",
           "isc_status_str", "isc_version")


class IscError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s: %s (%s)" % (where, STATUS.get(status, status),
                                          status_str(status)))


THRESHOLD_CROSSOVER = -1.0  # ISC_THRESHOLD_CROSSOVER: AUTO's per-shape crossover

KERNEL_IDS = {"none": 0, "fused": 1, "resident": 2, "ring": 3, "generic": 4, "fused_ring": 5, "fused_reg": 6}


class Tuning(ctypes.Structure):
    """isc_tuning: per-call plan overrides (0 = the library chooses)."""
    _fields_ = [(n, ctypes.c_int32) for n in ("kernel", "rows", "cols", "maps_per_lane", "phases", "waves",
                                               "wide_loads", "gemm_split", "reserved")]


class Plan(ctypes.Structure):
    """isc_plan: the sparse path's kernel and launch shape for a descriptor."""
    _fields_ = [("kernel", ctypes.c_int32), ("rows", ctypes.c_int32), ("cols", ctypes.c_int32),
                ("maps_per_lane", ctypes.c_int32), ("phases", ctypes.c_int32), ("waves", ctypes.c_int32),
                ("workgroups", ctypes.c_int64)]

    def asdict(self):
        d = {f: getattr(self, f) for f, _ in self._fields_}
        d["kernel"] = KERNEL_NAMES.get(d["kernel"], d["kernel"])
        return d


def tuning(**kw):
    """A Tuning from keyword fields; kernel may be a name ("fused_reg", ...)."""
    if "kernel" in kw and isinstance(kw["kernel"], str):
        kw["kernel"] = KERNEL_IDS[kw["kernel"]]
    return Tuning(**kw)


def _tuning_ref(t):
    if t is None:
        return None
    if isinstance(t, dict):
        t = tuning(**t)
    return ctypes.byref(t)


class ConvDesc(ctypes.Structure):
    """isc_conv_desc: Tab. 1 parameters plus the batch."""
    _fields_ = [(n, ctypes.c_int32) for n in ("N", "C", "H", "W", "K", "R", "S", "stride", "pad")]

    def astuple(self):
        return tuple(getattr(self, f) for f, _ in self._fields_)


_lib = None


def lib():
    """The loaded libisc.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libisc.so is not built (%s); run "
                          "`python -m paper_1704_07724_amd.build`" % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    i32, i64, sz, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p
    dp = ctypes.POINTER(ConvDesc)
    L.isc_out_shape.argtypes = [dp, ctypes.POINTER(i32), ctypes.POINTER(i32)]
    L.isc_workspace_size.argtypes = [dp, i32, ctypes.POINTER(sz)]
    tp = ctypes.POINTER(Tuning)
    L.isc_conv2d.argtypes = [dp, vp, vp, vp, vp, sz, i32, ctypes.c_float, vp]
    L.isc_conv2d_tuned.argtypes = [dp, vp, vp, vp, vp, sz, i32, ctypes.c_float, tp, vp]
    L.isc_decision.argtypes = [dp, vp, sz, ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(i32), vp]
    L.isc_conv2d_noalloc.argtypes = [dp, vp, vp, vp, i32, ctypes.c_float, vp]
    L.isc_crossover_sparsity.argtypes = [dp, ctypes.POINTER(ctypes.c_double)]
    L.isc_read_decision.argtypes = [vp, ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_uint64)]
    L.isc_sparse_plan.argtypes = [dp, tp, ctypes.POINTER(Plan)]
    L.isc_compact.argtypes = [dp, vp, vp, vp, vp, vp]
    L.isc_repacked_filter_size.argtypes = [dp, ctypes.POINTER(sz)]
    L.isc_repack_filter.argtypes = [dp, vp, vp, vp]
    L.isc_sparse_conv.argtypes = [dp, vp, vp, vp, vp, tp, vp]
    L.isc_im2col.argtypes = [dp, vp, vp, i64, vp]
    L.isc_gemm_f32.argtypes = [i32, i32, i32, vp, i64, vp, i64, vp, i64, vp]
    L.isc_sparse_conv_fused.argtypes = [dp, vp, vp, vp, tp, vp]
    L.isc_sparse_kernel.argtypes = [dp, ctypes.POINTER(i32)]
    L.isc_census_size.argtypes = [dp, ctypes.POINTER(sz)]
    L.isc_conv2d_relu.argtypes = [dp, vp, vp, sz, vp, vp, vp, vp, sz, vp, sz, i32, ctypes.c_float, tp, vp]
    L.isc_census_read.argtypes = [vp, sz, ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_uint64), vp]
    L.isc_conv2d_dw_workspace_size.argtypes = [dp, ctypes.POINTER(sz)]
    L.isc_conv2d_dw.argtypes = [dp, vp, vp, vp, vp, sz, tp, vp]
    for name in EXPORTS[:-2]:
        getattr(L, name).restype = ctypes.c_int
    L.isc_status_str.argtypes = [ctypes.c_int]
    L.isc_status_str.restype = ctypes.c_char_p
    L.isc_version.argtypes = []
    L.isc_version.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(status: int, where: str) -> None:
    if status != ISC_OK:
        raise IscError(status, where)


def status_str(status: int) -> str:
    return lib().isc_status_str(int(status)).decode()


isc_status_str = status_str


def isc_version() -> str:
    return lib().isc_version().decode()


def make_desc(N, C, H, W, K, R, S, stride=1, pad=0) -> ConvDesc:
    return ConvDesc(N, C, H, W, K, R, S, stride, pad)


def _desc_of(x_shape, w_shape, stride, pad) -> ConvDesc:
    N, C, H, W = (int(v) for v in x_shape)
    K, C2, R, S = (int(v) for v in w_shape)
    if C != C2:
        raise ValueError("input has %d channels, filter expects %d" % (C, C2))
    return make_desc(N, C, H, W, K, R, S, int(stride), int(pad))


def isc_out_shape(desc: ConvDesc):
    ho, wo = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().isc_out_shape(ctypes.byref(desc), ctypes.byref(ho), ctypes.byref(wo)),
           "isc_out_shape")
    return ho.value, wo.value


def isc_workspace_size(desc: ConvDesc, path="auto") -> int:
    n = ctypes.c_size_t()
    _check(lib().isc_workspace_size(ctypes.byref(desc), _path(path), ctypes.byref(n)),
           "isc_workspace_size")
    return n.value


def _path(path) -> int:
    if isinstance(path, str):
        return PATHS[path]
    return int(path)


def _torch():
    import torch
    return torch


def _stream(stream):
    torch = _torch()
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _on(stream):
    """Context in which the call's temporaries are allocated: the caller's
    stream when one is given (so that the caching allocator keeps them for
    that stream), else the current one."""
    if stream is None:
        return contextlib.nullcontext()
    torch = _torch()
    if not isinstance(stream, torch.cuda.Stream):
        stream = torch.cuda.ExternalStream(int(stream))
    return torch.cuda.stream(stream)


def default_path(path=None):
    """The path of a call: the argument, else ISC_PATH, else "auto"."""
    if path is None:
        path = os.environ.get("ISC_PATH", "auto") or "auto"
    return path


def default_threshold(threshold=None):
    """AUTO's threshold: the argument, else ISC_SPARSE_THRESHOLD, else the
    library's per-shape crossover (THRESHOLD_CROSSOVER)."""
    if threshold is None:
        env = os.environ.get("ISC_SPARSE_THRESHOLD")
        threshold = float(env) if env else THRESHOLD_CROSSOVER
    return float(threshold)


def _dev_f32(t, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.float32:
        raise TypeError("%s must be a float32 CUDA/HIP tensor" % name)
    return t.contiguous()


def workspace(desc: ConvDesc, path="auto", device=None):
    """A device workspace of isc_workspace_size bytes (256-byte aligned)."""
    torch = _torch()
    n = isc_workspace_size(desc, path)
    return torch.empty(max(n, 1), dtype=torch.uint8, device=device or "cuda")


def isc_conv2d(x, w, stride=1, pad=0, path=None, threshold=None, out=None, ws=None,
               stream=None, tuning=None):
    """y = conv(x, w) (Eq. 1 with batch, stride, zero padding) on the GPU.

    x: [N, C, H, W] float32, w: [K, C, R, S] float32 (device tensors).
    path: "auto" | "sparse" | "dense" (default: ISC_PATH or "auto");
    threshold: sparsity at or above which "auto" takes the sparse path
    (default: ISC_SPARSE_THRESHOLD, else the per-shape crossover);
    tuning: plan overrides (a Tuning or a dict of its fields).  Returns y
    [N, K, Ho, Wo] (``out`` if given).
    """
    torch = _torch()
    path = default_path(path)
    threshold = default_threshold(threshold)
    with _on(stream):
        x = _dev_f32(x, "x")
        w = _dev_f32(w, "w")
        desc = _desc_of(x.shape, w.shape, stride, pad)
        ho, wo = isc_out_shape(desc)
        if out is None:
            out = torch.empty((desc.N, desc.K, ho, wo), dtype=torch.float32, device=x.device)
        elif not out.is_contiguous() or tuple(out.shape) != (desc.N, desc.K, ho, wo):
            raise ValueError("out must be a contiguous [N, K, Ho, Wo] tensor")
        if ws is None:
            ws = workspace(desc, path, x.device)
        if tuning is None:
            st = lib().isc_conv2d(ctypes.byref(desc), x.data_ptr(), w.data_ptr(), out.data_ptr(),
                                  ws.data_ptr(), _nbytes(ws), _path(path), threshold, _stream(stream))
        else:
            st = lib().isc_conv2d_tuned(ctypes.byref(desc), x.data_ptr(), w.data_ptr(), out.data_ptr(),
                                        ws.data_ptr(), _nbytes(ws), _path(path), threshold,
                                        _tuning_ref(tuning), _stream(stream))
        _check(st, "isc_conv2d")
    return out


NOALLOC_SCRATCH_BYTES = 16 << 20  # ISC_NOALLOC_SCRATCH_BYTES


def isc_conv2d_noalloc(x, w, out, stride=1, pad=0, path=None, threshold=None, stream=None):
    """isc_conv2d with the library's own per-device scratch as workspace: the
    C call allocates nothing (x, w and out are the caller's device tensors,
    all contiguous).  Calls that overlap in time on one GPU race."""
    torch = _torch()
    for t, name in ((x, "x"), (w, "w"), (out, "out")):
        if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.float32 or not t.is_contiguous():
            raise TypeError("%s must be a contiguous float32 CUDA/HIP tensor" % name)
    desc = _desc_of(x.shape, w.shape, stride, pad)
    ho, wo = isc_out_shape(desc)
    if tuple(out.shape) != (desc.N, desc.K, ho, wo):
        raise ValueError("out must be [N, K, Ho, Wo]")
    _check(lib().isc_conv2d_noalloc(ctypes.byref(desc), x.data_ptr(), w.data_ptr(), out.data_ptr(),
                                    _path(default_path(path)), default_threshold(threshold), _stream(stream)),
           "isc_conv2d_noalloc")
    return out


def isc_read_decision(ws):
    """(path_name, nnz) from the workspace record, read by the host; the
    caller has synchronised the call that wrote it."""
    nnz = ctypes.c_uint64()
    path = ctypes.c_int32()
    _check(lib().isc_read_decision(ws.data_ptr(), ctypes.byref(path), ctypes.byref(nnz)), "isc_read_decision")
    return PATH_NAMES.get(path.value, path.value), nnz.value


def isc_decision(desc: ConvDesc, ws, stream=None):
    """(nnz_total, path_name) recorded by the last isc_conv2d on ``ws``;
    synchronises the stream."""
    nnz = ctypes.c_uint64()
    path = ctypes.c_int32()
    _check(lib().isc_decision(ctypes.byref(desc), ws.data_ptr(), ws.numel() * ws.element_size(),
                              ctypes.byref(nnz), ctypes.byref(path), _stream(stream)),
           "isc_decision")
    return nnz.value, PATH_NAMES.get(path.value, path.value)


def isc_census_size(desc: ConvDesc) -> int:
    n = ctypes.c_size_t()
    _check(lib().isc_census_size(ctypes.byref(desc), ctypes.byref(n)), "isc_census_size")
    return n.value


def census(desc: ConvDesc, device=None):
    """A device buffer for the census of the output of the layer `desc`
    (isc_census_size bytes; torch's allocations are 256-byte aligned)."""
    torch = _torch()
    return torch.empty(isc_census_size(desc), dtype=torch.uint8, device=device or "cuda")


def _nbytes(t):
    return t.numel() * t.element_size()


def isc_conv2d_relu(x, w, stride=1, pad=0, path=None, threshold=None, x_census=None, wt=None,
                    y_census=None, out=None, ws=None, stream=None, tuning=None):
    """y = max(0, conv(x, w)) (Eq. 1, then the rectifier of Eq. 2) with the
    nonzero count of y written to ``y_census`` (a buffer from ``census``)
    when given.  ``x_census``: the census of x from the call that wrote x
    (AUTO then decides from it instead of counting x).  ``wt``: a
    RepackedFilter of w (else w is repacked in the workspace).  path,
    threshold, tuning: as for isc_conv2d.  Returns y."""
    torch = _torch()
    path = default_path(path)
    threshold = default_threshold(threshold)
    with _on(stream):
        x = _dev_f32(x, "x")
        w = _dev_f32(w, "w")
        desc = _desc_of(x.shape, w.shape, stride, pad)
        ho, wo = isc_out_shape(desc)
        if out is None:
            out = torch.empty((desc.N, desc.K, ho, wo), dtype=torch.float32, device=x.device)
        elif not out.is_contiguous() or tuple(out.shape) != (desc.N, desc.K, ho, wo):
            raise ValueError("out must be a contiguous [N, K, Ho, Wo] tensor")
        if ws is None:
            ws = workspace(desc, path, x.device)
        if wt is not None and (wt.K, wt.C, wt.R, wt.S) != tuple(int(v) for v in w.shape):
            raise ValueError("repacked filter does not match w")
        _check(lib().isc_conv2d_relu(
            ctypes.byref(desc), x.data_ptr(),
            None if x_census is None else x_census.data_ptr(), 0 if x_census is None else _nbytes(x_census),
            w.data_ptr(), None if wt is None else wt.data.data_ptr(), out.data_ptr(),
            None if y_census is None else y_census.data_ptr(), 0 if y_census is None else _nbytes(y_census),
            ws.data_ptr(), _nbytes(ws), _path(path), threshold, _tuning_ref(tuning), _stream(stream)),
            "isc_conv2d_relu")
    return out


def isc_census_read(census_buf, stream=None):
    """(entries covered, nonzero count) of a census; synchronises the stream."""
    elems = ctypes.c_uint64()
    nnz = ctypes.c_uint64()
    _check(lib().isc_census_read(census_buf.data_ptr(), _nbytes(census_buf), ctypes.byref(elems),
                                 ctypes.byref(nnz), _stream(stream)), "isc_census_read")
    return elems.value, nnz.value


def isc_conv2d_dw_workspace_size(desc: ConvDesc) -> int:
    n = ctypes.c_size_t()
    _check(lib().isc_conv2d_dw_workspace_size(ctypes.byref(desc), ctypes.byref(n)), "isc_conv2d_dw_workspace_size")
    return n.value


def isc_conv2d_dw(x, dy, R, S, stride=1, pad=0, out=None, ws=None, stream=None, tuning=None):
    """The weight gradient dw [K, C, R, S] of Eq. 1 from x [N, C, H, W] and
    the output gradient dy [N, K, Ho, Wo], over the nonzero inputs only."""
    torch = _torch()
    with _on(stream):
        x = _dev_f32(x, "x")
        dy = _dev_f32(dy, "dy")
        N, C, H, W = (int(v) for v in x.shape)
        K = int(dy.shape[1])
        desc = make_desc(N, C, H, W, K, int(R), int(S), int(stride), int(pad))
        ho, wo = isc_out_shape(desc)
        if tuple(dy.shape) != (N, K, ho, wo):
            raise ValueError("dy must be [N, K, Ho, Wo] = %r" % ((N, K, ho, wo),))
        if out is None:
            out = torch.empty((K, C, int(R), int(S)), dtype=torch.float32, device=x.device)
        elif not out.is_contiguous() or tuple(out.shape) != (K, C, int(R), int(S)):
            raise ValueError("out must be a contiguous [K, C, R, S] tensor")
        if ws is None:
            ws = torch.empty(max(isc_conv2d_dw_workspace_size(desc), 1), dtype=torch.uint8, device=x.device)
        _check(lib().isc_conv2d_dw(ctypes.byref(desc), x.data_ptr(), dy.data_ptr(), out.data_ptr(), ws.data_ptr(),
                                   _nbytes(ws), _tuning_ref(tuning), _stream(stream)), "isc_conv2d_dw")
    return out


NZ_TAIL = 256  # spare entries isc_sparse_conv may read past the last plane


def isc_compact(x, stream=None, out=None):
    """ISC step 1 on the GPU.

    Returns (row_ptr [N*C, H+1] int32, entries [N*C, H*W, 2] int32 holding
    (value bits, (row << 16) | column), nnz_total [1] int64), all on the
    device; entries past a plane's count are left as allocated (zeros here).
    The entries view sits in a buffer with NZ_TAIL spare entries, so it can
    be passed to isc_sparse_conv.  ``out`` reuses (row_ptr, entries, total).
    """
    torch = _torch()
    with _on(stream):
        x = _dev_f32(x, "x")
        N, C, H, W = (int(v) for v in x.shape)
        desc = make_desc(N, C, H, W, 1, 1, 1, 1, 0)
        if out is None:
            row_ptr = torch.empty((N * C, H + 1), dtype=torch.int32, device=x.device)
            buf = torch.zeros((N * C * H * W + NZ_TAIL, 2), dtype=torch.int32, device=x.device)
            nz = buf[:N * C * H * W].view(N * C, H * W, 2)
            total = torch.empty(1, dtype=torch.int64, device=x.device)
        else:
            row_ptr, nz, total = out
        _check(lib().isc_compact(ctypes.byref(desc), x.data_ptr(), row_ptr.data_ptr(), nz.data_ptr(),
                                 total.data_ptr(), _stream(stream)), "isc_compact")
    return row_ptr, nz, total


def isc_repacked_filter_size(desc: ConvDesc) -> int:
    n = ctypes.c_size_t()
    _check(lib().isc_repacked_filter_size(ctypes.byref(desc), ctypes.byref(n)),
           "isc_repacked_filter_size")
    return n.value


class RepackedFilter:
    """ISC step 2's blocked K-contiguous filter (see isc_repack_filter)."""

    def __init__(self, data, K, C, R, S):
        self.data, self.K, self.C, self.R, self.S = data, K, C, R, S

    def dense(self):
        """[C, R, S, Kp] view of the buffer (Kp = K rounded up to 64)."""
        kp = (self.K + 63) // 64 * 64
        return self.data.view(self.C, self.R, self.S, kp)


def isc_repack_filter(w, out=None, stream=None):
    """ISC step 2's filter layout for w [K, C, R, S] (a RepackedFilter)."""
    torch = _torch()
    with _on(stream):
        w = _dev_f32(w, "w")
        K, C, R, S = (int(v) for v in w.shape)
        desc = make_desc(1, C, R, S, K, R, S, 1, 0)
        n = isc_repacked_filter_size(desc) // 4
        data = out if out is not None else torch.empty(n, dtype=torch.float32, device=w.device)
        _check(lib().isc_repack_filter(ctypes.byref(desc), w.data_ptr(), data.data_ptr(),
                                       _stream(stream)), "isc_repack_filter")
    return RepackedFilter(data, K, C, R, S)


KERNEL_NAMES = {0: "none", 1: "fused", 2: "resident", 3: "ring", 4: "generic", 5: "fused_ring", 6: "fused_reg"}


def isc_sparse_kernel(desc: ConvDesc, tuning=None) -> str:
    """Which kernel isc_conv2d's sparse path runs for desc (under the given
    overrides): "fused", "fused_reg", "fused_ring" (on-the-fly compaction),
    "resident", "ring" or "generic" (over compacted lists), or "none"."""
    if tuning is not None:
        return isc_sparse_plan(desc, tuning)["kernel"]
    which = ctypes.c_int32(-1)
    _check(lib().isc_sparse_kernel(ctypes.byref(desc), ctypes.byref(which)), "isc_sparse_kernel")
    return KERNEL_NAMES[which.value]


def isc_crossover_sparsity(desc: ConvDesc) -> float:
    """The sparsity at or above which AUTO (per-shape crossover) takes the
    sparse path for desc; 2.0 when it never does."""
    v = ctypes.c_double()
    _check(lib().isc_crossover_sparsity(ctypes.byref(desc), ctypes.byref(v)), "isc_crossover_sparsity")
    return v.value


def isc_sparse_plan(desc: ConvDesc, tuning=None) -> dict:
    """The sparse path's plan for desc: kernel, rows, cols, maps_per_lane,
    phases, waves, workgroups."""
    p = Plan()
    _check(lib().isc_sparse_plan(ctypes.byref(desc), _tuning_ref(tuning), ctypes.byref(p)), "isc_sparse_plan")
    return p.asdict()


def isc_sparse_conv_fused(x, wt, stride=1, pad=0, out=None, stream=None, tuning=None):
    """ISC steps 1-3 in one launch (compaction on the fly) with a
    RepackedFilter (isc_repack_filter), no workspace; returns y [N, K, Ho,
    Wo].  Raises IscError (LIMIT) for shapes the kernel does not take."""
    torch = _torch()
    with _on(stream):
        x = _dev_f32(x, "x")
        N, C, H, W = (int(v) for v in x.shape)
        K, R, S = wt.K, wt.R, wt.S
        if C != wt.C:
            raise ValueError("channel mismatch")
        desc = make_desc(N, C, H, W, K, R, S, int(stride), int(pad))
        ho, wo = isc_out_shape(desc)
        if out is None:
            out = torch.empty((N, K, ho, wo), dtype=torch.float32, device=x.device)
        elif not out.is_contiguous() or tuple(out.shape) != (N, K, ho, wo):
            raise ValueError("out must be a contiguous [N, K, Ho, Wo] tensor")
        _check(lib().isc_sparse_conv_fused(ctypes.byref(desc), x.data_ptr(), wt.data.data_ptr(), out.data_ptr(),
                                           _tuning_ref(tuning), _stream(stream)), "isc_sparse_conv_fused")
    return out


def isc_sparse_conv(x_shape, lists, wt, stride=1, pad=0, out=None, stream=None, tuning=None):
    """ISC steps 2-3 from compacted lists (isc_compact's (row_ptr, entries,
    ...)) and a RepackedFilter; returns y [N, K, Ho, Wo]."""
    torch = _torch()
    N, C, H, W = (int(v) for v in x_shape)
    K, R, S = wt.K, wt.R, wt.S
    if C != wt.C:
        raise ValueError("channel mismatch")
    row_ptr, nz = lists[0], lists[1]
    desc = make_desc(N, C, H, W, K, R, S, int(stride), int(pad))
    ho, wo = isc_out_shape(desc)
    with _on(stream):
        if out is None:
            out = torch.empty((N, K, ho, wo), dtype=torch.float32, device=wt.data.device)
        _check(lib().isc_sparse_conv(ctypes.byref(desc), row_ptr.data_ptr(), nz.data_ptr(),
                                     wt.data.data_ptr(), out.data_ptr(), _tuning_ref(tuning), _stream(stream)),
               "isc_sparse_conv")
    return out


def isc_im2col(x, R, S, stride=1, pad=0, ldc=None, out=None, stream=None):
    """The unrolled input matrix M_I (Fig. 3) on the GPU: [C*R*S, ldc] float32
    (written into `out` when given: contiguous, that shape)."""
    torch = _torch()
    with _on(stream):
        return _im2col(torch, x, R, S, stride, pad, ldc, out, stream)


def _im2col(torch, x, R, S, stride, pad, ldc, out, stream):
    x = _dev_f32(x, "x")
    N, C, H, W = (int(v) for v in x.shape)
    desc = make_desc(N, C, H, W, 1, int(R), int(S), int(stride), int(pad))
    ho, wo = isc_out_shape(desc)
    ldc = N * ho * wo if ldc is None else int(ldc)
    if out is None:
        col = torch.empty((C * R * S, ldc), dtype=torch.float32, device=x.device)
    else:
        col = out
        if (not isinstance(col, torch.Tensor) or col.dtype != torch.float32 or not col.is_contiguous()
                or tuple(col.shape) != (C * R * S, ldc) or col.device != x.device):
            raise ValueError("out must be a contiguous float32 [C*R*S, ldc] tensor on x's device")
    _check(lib().isc_im2col(ctypes.byref(desc), x.data_ptr(), col.data_ptr(), ldc,
                            _stream(stream)), "isc_im2col")
    return col


def isc_gemm_f32(a, b, out=None, stream=None):
    """c = a @ b on the fp32 matrix cores (a [M, Kd], b [Kd, N], row-major)."""
    torch = _torch()
    with _on(stream):
        return _gemm(torch, a, b, out, stream)


def _gemm(torch, a, b, out, stream):
    a = _dev_f32(a, "a")
    b = _dev_f32(b, "b")
    M, Kd = (int(v) for v in a.shape)
    Kd2, N = (int(v) for v in b.shape)
    if Kd != Kd2:
        raise ValueError("inner dimensions differ")
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=a.device)
    _check(lib().isc_gemm_f32(M, N, Kd, a.data_ptr(), Kd, b.data_ptr(), N, out.data_ptr(), N,
                              _stream(stream)), "isc_gemm_f32")
    return out
