// C ABI of the library (include/isc.h): argument validation on the host,
// workspace layout, and the launch sequences of the sparse path (ISC steps
// 1-3), the dense path (Fig. 3) and the dispatcher between them.
#include "isc.h"
#include "isc_internal.hpp"

#include <atomic>
#include <cmath>
#include <cstring>
#include <algorithm>
#include <limits>
#include <vector>

namespace isc {
bool sparse_conv_feasible(const SparseShape &sh);
}

namespace {

using isc::Ctrl;
using isc::NzEntry;

constexpr int64_t kI32Max = std::numeric_limits<int32_t>::max();
constexpr size_t kAlign = 256;
constexpr int64_t kColPad = 256;   // im2col rows padded to this many columns
constexpr int64_t kNzTail = 256;   // spare list entries after the last plane (read, never used)

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct Shape {
    int64_t N, C, H, W, K, R, S, T, P, Ho, Wo;
    int64_t in_elems() const { return N * C * H * W; }
    int64_t out_elems() const { return N * K * Ho * Wo; }
    int64_t filt_elems() const { return K * C * R * S; }
    int64_t crs() const { return C * R * S; }
    int64_t ncols() const { return N * Ho * Wo; }
    int64_t ldcol() const { return (ncols() + kColPad - 1) / kColPad * kColPad; }
};

int64_t out_extent(int64_t in, int64_t k, int64_t pad, int64_t stride) {
    const int64_t num = in + 2 * pad - k;
    if (num < 0) return 0;
    return num / stride + 1;
}

int check_desc(const isc_conv_desc *d, Shape *sh) {
    if (!d) return ISC_ERR_NULL;
    if (d->N < 1 || d->C < 1 || d->H < 1 || d->W < 1 || d->K < 1 || d->R < 1 || d->S < 1 ||
        d->stride < 1 || d->pad < 0)
        return ISC_ERR_SHAPE;
    Shape s{d->N, d->C, d->H, d->W, d->K, d->R, d->S, d->stride, d->pad, 0, 0};
    s.Ho = out_extent(s.H, s.R, s.P, s.T);
    s.Wo = out_extent(s.W, s.S, s.P, s.T);
    if (s.Ho < 1 || s.Wo < 1) return ISC_ERR_SHAPE;
    if (s.H > 65535 || s.W > 65535) return ISC_ERR_LIMIT;
    if (s.in_elems() > kI32Max || s.out_elems() > kI32Max || s.filt_elems() > kI32Max ||
        s.ncols() > kI32Max || s.Ho > kI32Max || s.Wo > kI32Max)
        return ISC_ERR_LIMIT;
    // the dense path materialises the im2col matrix only when C*R*S >= 2^16
    if (!isc::conv_gemm_implicit_ok(static_cast<int>(s.C), static_cast<int>(s.R), static_cast<int>(s.S)) &&
        s.crs() * s.ldcol() > kI32Max)
        return ISC_ERR_LIMIT;
    if ((s.K + 31) / 32 > 65535) return ISC_ERR_LIMIT;  // GEMM grid rows
    *sh = s;
    return ISC_OK;
}

bool valid_path(int32_t p) { return p == ISC_PATH_AUTO || p == ISC_PATH_SPARSE || p == ISC_PATH_DENSE; }

isc::SparseShape sparse_shape(const Shape &s, const isc_tuning *tu = nullptr) {
    return isc::SparseShape{static_cast<int>(s.N),  static_cast<int>(s.C), static_cast<int>(s.H),
                            static_cast<int>(s.W),  static_cast<int>(s.K), static_cast<int>(s.R),
                            static_cast<int>(s.S),  static_cast<int>(s.T), static_cast<int>(s.P),
                            static_cast<int>(s.Ho), static_cast<int>(s.Wo), tu ? *tu : isc_tuning{}};
}

// A caller's overrides are well formed (the reserved field is zero).
bool tuning_ok(const isc_tuning *tu) { return tu == nullptr || tu->reserved == 0; }

struct Layout {
    size_t ctrl = 0, parts = 0, row_ptr = 0, nz = 0, wt = 0, col = 0, split = 0, total = 0;
    bool sparse = false, dense = false;
    bool implicit = false;  // dense path gathers im2col inside the GEMM (no col buffer)
    bool fused = false;     // sparse path compacts on the fly (no lists; the repacked filter only)
};

// split: room for the dense GEMM's split reduction when it takes one (a
// caller's tuning gemm_split = -1 turns the split off and needs none).
Layout layout_for(const Shape &s, int32_t path, bool split_ok = true) {
    Layout L;
    L.sparse = path != ISC_PATH_DENSE;
    L.dense = path != ISC_PATH_SPARSE;
    size_t off = align_up(sizeof(Ctrl), kAlign);
    L.fused = isc::sparse_fused_applies(sparse_shape(s));
    if (L.sparse) {
        L.parts = off;
        off = align_up(off + sizeof(uint32_t) * isc::kMaxParts, kAlign);
    }
    if (L.sparse && !L.fused) {
        L.row_ptr = off;
        off = align_up(off + sizeof(int32_t) * static_cast<size_t>(s.N * s.C * (s.H + 1)), kAlign);
        L.nz = off;
        off = align_up(off + sizeof(NzEntry) * static_cast<size_t>(s.in_elems() + kNzTail), kAlign);
    }
    if (L.sparse) {
        L.wt = off;
        off = align_up(off + sizeof(float) * isc::repacked_filter_floats(static_cast<int>(s.K), static_cast<int>(s.C),
                                                                         static_cast<int>(s.R), static_cast<int>(s.S)),
                       kAlign);
    }
    L.implicit = isc::conv_gemm_implicit_ok(static_cast<int>(s.C), static_cast<int>(s.R), static_cast<int>(s.S));
    if (L.dense && !L.implicit) {
        L.col = off;
        off = align_up(off + sizeof(float) * static_cast<size_t>(s.crs() * s.ldcol()), kAlign);
    }
    // the partial sums of the implicit GEMM's split reduction (last, so the
    // layout without it is a prefix of the layout with it)
    const size_t split = split_ok && L.dense && L.implicit
                             ? isc::conv_gemm_split_floats(static_cast<int>(s.K), s.ncols(), static_cast<int>(s.crs()))
                             : 0;
    if (split > 0) {
        L.split = off;
        off = align_up(off + sizeof(float) * split, kAlign);
    }
    L.total = off;
    return L;
}

bool aligned(const void *p, size_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; }

bool overlap(const void *a, size_t an, const void *b, size_t bn) {
    const uintptr_t x0 = reinterpret_cast<uintptr_t>(a), y0 = reinterpret_cast<uintptr_t>(b);
    return x0 < y0 + bn && y0 < x0 + an;
}

// The current device must be a gfx950.  The answer is kept per device id:
// the architecture of a device cannot change while the process runs, and
// asking the runtime for the device's properties on every launch would add
// host time to every call.  This memo is the library's only state besides
// the per-kernel LDS-size grants (hipFuncSetAttribute is asked once per
// kernel) and, for the allocation-free entry point, each device's scratch
// address.
int check_device() {
    static std::atomic<int> state[64];  // 0 unknown, 1 gfx950, 2 other
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return ISC_ERR_DEVICE;
    if (dev < 64) {
        const int st = state[dev].load(std::memory_order_relaxed);
        if (st == 1) return ISC_OK;
        if (st == 2) return ISC_ERR_DEVICE;
    }
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return ISC_ERR_DEVICE;
    const bool ok = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    if (dev < 64) state[dev].store(ok ? 1 : 2, std::memory_order_relaxed);
    return ok ? ISC_OK : ISC_ERR_DEVICE;
}

// Largest nonzero count n with 1 - n/total >= threshold (the sparsity test of
// the dispatcher, evaluated in double exactly as written).
long long nnz_limit_for(int64_t total, float threshold) {
    const double th = static_cast<double>(threshold);
    auto sparse_enough = [&](int64_t n) {
        return 1.0 - static_cast<double>(n) / static_cast<double>(total) >= th;
    };
    int64_t n = static_cast<int64_t>(std::floor((1.0 - th) * static_cast<double>(total)));
    n = std::max<int64_t>(-1, std::min<int64_t>(n, total));
    while (n + 1 <= total && sparse_enough(n + 1)) ++n;
    while (n >= 0 && !sparse_enough(n)) --n;
    return static_cast<long long>(n);  // -1 only for a threshold above 1 (rejected)
}

int hip_status(hipError_t e) { return e == hipSuccess ? ISC_OK : ISC_ERR_HIP; }

// Workspace of isc_conv2d_noalloc: a device array each GPU holds until the
// process ends.  In host code its name is a host-side stand-in, not a device
// address; the device address comes from hipGetSymbolAddress, once per
// device with that device current, and only that address is ever handed to
// a kernel or a copy.
constexpr size_t kScratchBytes = ISC_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::atomic<void *> scratch_addr[kMaxDevices];

// The current device's scratch address, looked up on the first call on the
// device (ISC_ERR_DEVICE or ISC_ERR_HIP on failure).
int scratch_for_current_device(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return ISC_ERR_DEVICE;
    void *p = scratch_addr[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return ISC_ERR_HIP;
        scratch_addr[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return ISC_OK;
}

// What isc_conv2d_relu adds to isc_conv2d: the epilogue (rectifier and
// census of y), the census of x, and a caller's repacked filter.
struct Chain {
    const isc::CensusHeader *x_census = nullptr;
    uint32_t x_cap = 0;
    size_t x_census_bytes = 0;
    size_t y_census_bytes = 0;
    const float *wt = nullptr;
    isc::Epilogue epi{};
};

uint32_t census_cap(size_t bytes) {
    const size_t n = (bytes - sizeof(isc::CensusHeader)) / sizeof(uint32_t);
    return static_cast<uint32_t>(std::min<size_t>(n, std::numeric_limits<uint32_t>::max()) / 4 * 4);
}

// A census has room for the workgroups of every kernel that may write the
// output: the on-the-fly sparse kernels, the stand-alone epilogue pass
// after the list kernels, and the GEMM.
size_t census_bytes(const Shape &s) {
    const int64_t groups = std::max<int64_t>({isc::sparse_fused_max_groups(sparse_shape(s)),
                                              static_cast<int64_t>(isc::kRectifyGroups),
                                              isc::gemm_max_groups(s.K, s.ncols())});
    return sizeof(isc::CensusHeader) + sizeof(uint32_t) * isc::census_slots_for(groups);
}

int conv_impl(const isc_conv_desc *d, const float *x, const float *w, float *y, void *ws, size_t ws_bytes,
              int32_t path, float threshold, void *stream, const Chain *ch, const isc_tuning *tu) {
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    if (!x || !w || !y || !ws) return ISC_ERR_NULL;
    if (!valid_path(path)) return ISC_ERR_PATH;
    if (!(threshold >= 0.0f && threshold <= 1.0f) && !(threshold < 0.0f)) return ISC_ERR_ARG;
    if (!tuning_ok(tu)) return ISC_ERR_ARG;
    if (!aligned(x, 4) || !aligned(w, 4) || !aligned(y, 4) || !aligned(ws, kAlign)) return ISC_ERR_ALIGN;
    const Layout L = layout_for(s, path, !(tu && tu->gemm_split < 0));
    if (ws_bytes < L.total) return ISC_ERR_WORKSPACE;
    const size_t xbytes = sizeof(float) * static_cast<size_t>(s.in_elems());
    const size_t ybytes = sizeof(float) * static_cast<size_t>(s.out_elems());
    const size_t wbytes = sizeof(float) * static_cast<size_t>(s.filt_elems());
    if (overlap(y, ybytes, x, xbytes) || overlap(y, ybytes, w, wbytes) || overlap(y, ybytes, ws, L.total))
        return ISC_ERR_ALIAS;
    const isc::Epilogue epi = ch ? ch->epi : isc::Epilogue{};
    if (ch) {
        const size_t tbytes = sizeof(float) * isc::repacked_filter_floats(static_cast<int>(s.K), static_cast<int>(s.C),
                                                                         static_cast<int>(s.R), static_cast<int>(s.S));
        const void *yc = epi.census;
        const size_t ycb = ch->y_census_bytes;
        if (ch->wt && (overlap(y, ybytes, ch->wt, tbytes) || overlap(ch->wt, tbytes, ws, L.total)))
            return ISC_ERR_ALIAS;
        if (ch->x_census && overlap(y, ybytes, ch->x_census, ch->x_census_bytes)) return ISC_ERR_ALIAS;
        if (yc && (overlap(yc, ycb, x, xbytes) || overlap(yc, ycb, y, ybytes) || overlap(yc, ycb, w, wbytes) ||
                   overlap(yc, ycb, ws, L.total) || (ch->wt && overlap(yc, ycb, ch->wt, tbytes)) ||
                   (ch->x_census && overlap(yc, ycb, ch->x_census, ch->x_census_bytes))))
            return ISC_ERR_ALIAS;
    }

    const isc::SparseShape sh = sparse_shape(s, tu);
    const bool sparse_fits = L.fused || isc::sparse_conv_feasible(sh);
    if (path == ISC_PATH_SPARSE && !sparse_fits) return ISC_ERR_LIMIT;
    if (path == ISC_PATH_AUTO && !sparse_fits) path = ISC_PATH_DENSE;  // dense buffers are in L

    st = check_device();
    if (st) return st;

    hipStream_t hs = static_cast<hipStream_t>(stream);
    char *base = static_cast<char *>(ws);
    Ctrl *ctrl = reinterpret_cast<Ctrl *>(base);
    hipError_t e = hipSuccess;
    uint32_t *parts = L.sparse ? reinterpret_cast<uint32_t *>(base + L.parts) : nullptr;
    int nparts = 0;
    const long long limit = threshold < 0.0f ? isc::crossover_nnz_limit(sh) : nnz_limit_for(s.in_elems(), threshold);
    // a limit no count can cross decides AUTO on the host: every count picks
    // the sparse path (the count still runs, for the record), or none does
    // (the dense path alone, as if asked for)
    if (path == ISC_PATH_AUTO && limit >= s.in_elems()) path = ISC_PATH_SPARSE;
    if (path == ISC_PATH_AUTO && limit < 0) path = ISC_PATH_DENSE;
    const int gate_sparse = path == ISC_PATH_AUTO ? isc::kGateIfSparse : isc::kGateAlways;

    if (path != ISC_PATH_DENSE) {
        // steps 2-3 are gated by the device-side decision in AUTO and record
        // the count and the path taken
        float *wt_ws = reinterpret_cast<float *>(base + L.wt);
        if (L.fused) {
            const float *wt = ch && ch->wt ? ch->wt : wt_ws;
            isc::Decision dec{parts, 0, limit, gate_sparse, ctrl};
            if (ch && ch->x_census) {
                // the count comes from the census of x, summed once into
                // the parts: no pass over x
                if (!ch->wt && (e = isc::launch_repack_filter(w, sh.K, sh.C, sh.R, sh.S, wt_ws, hs)) != hipSuccess)
                    return hip_status(e);
                // and a filter repacked by the caller, cold in cache, warmed
                // in the same launch (the fused kernels read it a channel
                // at a time, one dependent step after another)
                const size_t wt_bytes =
                    ch->wt ? isc::repacked_filter_floats(sh.K, sh.C, sh.R, sh.S) * sizeof(float) : 0;
                if ((e = isc::launch_census_parts(ch->x_census, ch->x_cap, static_cast<unsigned long long>(s.in_elems()),
                                                  parts, ch->wt, wt_bytes, ctrl, hs)) != hipSuccess)
                    return hip_status(e);
                dec.nparts = 4;
            } else {
                // the count for the decision and the filter repack to
                // K-contiguous in one launch (or, with a filter the caller
                // repacked, its cache warm-up), then steps 1-3 in one launch
                const bool repack = !(ch && ch->wt);
                const size_t wt_bytes =
                    repack ? 0 : isc::repacked_filter_floats(sh.K, sh.C, sh.R, sh.S) * sizeof(float);
                if ((e = isc::launch_count_parts(x, s.in_elems(), parts, &nparts, hs, repack ? w : nullptr, sh.K,
                                                 sh.C, sh.R, sh.S, repack ? wt_ws : nullptr, repack ? nullptr : ch->wt,
                                                 wt_bytes, ctrl)) != hipSuccess)
                    return hip_status(e);
                dec.nparts = nparts;
            }
            if ((e = isc::launch_sparse_fused(sh, x, wt, y, dec, hs, epi)) != hipSuccess) return hip_status(e);
        } else {
            int32_t *row_ptr = reinterpret_cast<int32_t *>(base + L.row_ptr);
            NzEntry *nz = reinterpret_cast<NzEntry *>(base + L.nz);
            // step 1 and the filter repack to K-contiguous, one launch
            if ((e = isc::launch_prep(x, static_cast<int>(s.N * s.C), sh.H, sh.W, row_ptr, nz, parts, &nparts, w,
                                      sh.K, sh.C, sh.R, sh.S, wt_ws, hs)) != hipSuccess)
                return hip_status(e);
            isc::Decision dec{parts, nparts, limit, gate_sparse, ctrl};
            if ((e = isc::launch_sparse_conv(sh, row_ptr, nz, wt_ws, y, dec, hs)) != hipSuccess)
                return hip_status(e);
            if (epi.relu || epi.census) {
                // the list kernels store y without the epilogue: a pass of its
                // own, run iff the sparse path was taken
                isc::Decision after{nullptr, 0, limit, isc::kGateIfSparse, nullptr, ctrl};
                if ((e = isc::launch_rectify(y, s.out_elems(), epi, after, hs)) != hipSuccess)
                    return hip_status(e);
            }
        }
    }
    if (path != ISC_PATH_SPARSE) {
        // AUTO: run iff the sparse kernel, launched before on this stream,
        // recorded the dense path; DENSE alone: no count, recorded as such
        isc::Decision dec{nullptr, 0, limit, path == ISC_PATH_AUTO ? isc::kGateIfDense : isc::kGateAlways,
                          path == ISC_PATH_DENSE ? ctrl : nullptr, path == ISC_PATH_AUTO ? ctrl : nullptr};
        if (L.implicit) {
            // one launch: the GEMM gathers the im2col matrix from x
            float *part = L.split ? reinterpret_cast<float *>(base + L.split) : nullptr;
            if ((e = isc::launch_conv_gemm(x, w, y, sh.N, sh.C, sh.H, sh.W, sh.K, sh.R, sh.S, sh.T, sh.P, sh.Ho,
                                           sh.Wo, dec, hs, epi, part)) != hipSuccess)
                return hip_status(e);
        } else {
            float *col = reinterpret_cast<float *>(base + L.col);
            if ((e = isc::launch_im2col(x, sh.N, sh.C, sh.H, sh.W, sh.R, sh.S, sh.T, sh.P, sh.Ho, sh.Wo, col,
                                        s.ldcol(), dec, hs)) != hipSuccess)
                return hip_status(e);
            dec.record = nullptr;
            if ((e = isc::launch_gemm_f32(sh.K, static_cast<int>(s.ncols()), static_cast<int>(s.crs()), w,
                                          s.crs(), col, s.ldcol(), y, 0, sh.Ho * sh.Wo, true, dec, hs, epi)) !=
                hipSuccess)
                return hip_status(e);
        }
    }
    return ISC_OK;
}

}  // namespace

extern "C" {

const char *isc_version(void) { return "isc-mi355x 0.1 (gfx950)"; }

const char *isc_status_str(int status) {
    switch (status) {
    case ISC_OK: return "ok";
    case ISC_ERR_NULL: return "null pointer";
    case ISC_ERR_SHAPE: return "invalid shape";
    case ISC_ERR_LIMIT: return "size limit exceeded";
    case ISC_ERR_WORKSPACE: return "workspace too small";
    case ISC_ERR_ALIAS: return "output overlaps an input or the workspace";
    case ISC_ERR_PATH: return "invalid path";
    case ISC_ERR_DEVICE: return "no gfx950 device";
    case ISC_ERR_HIP: return "HIP runtime error";
    case ISC_ERR_ALIGN: return "misaligned pointer";
    case ISC_ERR_ARG: return "invalid argument";
    default: return "unknown status";
    }
}

int isc_out_shape(const isc_conv_desc *d, int32_t *Ho, int32_t *Wo) {
    if (!d || !Ho || !Wo) return ISC_ERR_NULL;
    if (d->H < 1 || d->W < 1 || d->R < 1 || d->S < 1 || d->stride < 1 || d->pad < 0)
        return ISC_ERR_SHAPE;
    const int64_t ho = out_extent(d->H, d->R, d->pad, d->stride);
    const int64_t wo = out_extent(d->W, d->S, d->pad, d->stride);
    if (ho < 1 || wo < 1) return ISC_ERR_SHAPE;
    *Ho = static_cast<int32_t>(ho);
    *Wo = static_cast<int32_t>(wo);
    return ISC_OK;
}

int isc_workspace_size(const isc_conv_desc *d, int32_t path, size_t *bytes) {
    if (!bytes) return ISC_ERR_NULL;
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    if (!valid_path(path)) return ISC_ERR_PATH;
    *bytes = layout_for(s, path).total;
    return ISC_OK;
}

int isc_conv2d(const isc_conv_desc *d, const float *x, const float *w, float *y, void *ws,
               size_t ws_bytes, int32_t path, float threshold, void *stream) {
    return conv_impl(d, x, w, y, ws, ws_bytes, path, threshold, stream, nullptr, nullptr);
}

int isc_conv2d_noalloc(const isc_conv_desc *d, const float *x, const float *w, float *y, int32_t path,
                       float threshold, void *stream) {
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    if (!x || !w || !y) return ISC_ERR_NULL;
    if (!valid_path(path)) return ISC_ERR_PATH;
    // the dense GEMM's split reduction only where its partial sums fit too
    isc_tuning nosplit{};
    nosplit.gemm_split = -1;
    const isc_tuning *tu = nullptr;
    if (layout_for(s, path).total > kScratchBytes) {
        if (layout_for(s, path, false).total > kScratchBytes) return ISC_ERR_LIMIT;
        tu = &nosplit;
    }
    st = check_device();
    if (st) return st;
    void *ws = nullptr;
    st = scratch_for_current_device(&ws);
    if (st) return st;
    return conv_impl(d, x, w, y, ws, kScratchBytes, path, threshold, stream, nullptr, tu);
}

int isc_conv2d_tuned(const isc_conv_desc *d, const float *x, const float *w, float *y, void *ws,
                     size_t ws_bytes, int32_t path, float threshold, const isc_tuning *tuning, void *stream) {
    return conv_impl(d, x, w, y, ws, ws_bytes, path, threshold, stream, nullptr, tuning);
}

int isc_census_size(const isc_conv_desc *d, size_t *bytes) {
    if (!bytes) return ISC_ERR_NULL;
    Shape s;
    const int st = check_desc(d, &s);
    if (st) return st;
    *bytes = census_bytes(s);
    return ISC_OK;
}

int isc_conv2d_relu(const isc_conv_desc *d, const float *x, const void *x_census, size_t x_census_bytes,
                    const float *w, const float *wt, float *y, void *y_census, size_t y_census_bytes, void *ws,
                    size_t ws_bytes, int32_t path, float threshold, const isc_tuning *tuning, void *stream) {
    Shape s;
    const int st = check_desc(d, &s);
    if (st) return st;
    Chain ch;
    ch.wt = wt;
    ch.epi.relu = 1;
    ch.epi.elems = static_cast<unsigned long long>(s.out_elems());
    if (x_census) {
        if (!aligned(x_census, 16)) return ISC_ERR_ALIGN;
        if (x_census_bytes < sizeof(isc::CensusHeader)) return ISC_ERR_WORKSPACE;
        ch.x_census = static_cast<const isc::CensusHeader *>(x_census);
        ch.x_cap = census_cap(x_census_bytes);
        ch.x_census_bytes = x_census_bytes;
    }
    if (y_census) {
        if (!aligned(y_census, 16)) return ISC_ERR_ALIGN;
        if (y_census_bytes < census_bytes(s)) return ISC_ERR_WORKSPACE;
        ch.epi.census = static_cast<isc::CensusHeader *>(y_census);
        ch.epi.cap = census_cap(y_census_bytes);
        ch.y_census_bytes = y_census_bytes;
    }
    if (wt && !aligned(wt, 16)) return ISC_ERR_ALIGN;
    return conv_impl(d, x, w, y, ws, ws_bytes, path, threshold, stream, &ch, tuning);
}

int isc_census_read(const void *census, size_t bytes, uint64_t *elems, uint64_t *nnz, void *stream) {
    if (!census || !elems || !nnz) return ISC_ERR_NULL;
    if (bytes < sizeof(isc::CensusHeader)) return ISC_ERR_WORKSPACE;
    const int st = check_device();
    if (st) return st;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    isc::CensusHeader h;
    hipError_t e = hipMemcpyAsync(&h, census, sizeof(h), hipMemcpyDeviceToHost, hs);
    if (e == hipSuccess) e = hipStreamSynchronize(hs);
    if (e != hipSuccess) return ISC_ERR_HIP;
    if (h.nslots % 4 != 0 || h.nslots > census_cap(bytes)) return ISC_ERR_ARG;  // not a census
    std::vector<uint32_t> slots(h.nslots);
    if (h.nslots) {
        e = hipMemcpyAsync(slots.data(), static_cast<const isc::CensusHeader *>(census) + 1,
                           sizeof(uint32_t) * h.nslots, hipMemcpyDeviceToHost, hs);
        if (e == hipSuccess) e = hipStreamSynchronize(hs);
        if (e != hipSuccess) return ISC_ERR_HIP;
    }
    uint64_t total = 0;
    for (uint32_t v : slots) total += v;
    *elems = h.elems;
    *nnz = total;
    return ISC_OK;
}

int isc_sparse_conv_fused(const isc_conv_desc *d, const float *x, const float *wt, float *y,
                          const isc_tuning *tuning, void *stream) {
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    if (!x || !wt || !y) return ISC_ERR_NULL;
    if (!tuning_ok(tuning)) return ISC_ERR_ARG;
    if (!aligned(x, 4) || !aligned(wt, 4) || !aligned(y, 4)) return ISC_ERR_ALIGN;
    const isc::SparseShape sh = sparse_shape(s, tuning);
    if (!isc::sparse_fused_applies(sh)) return ISC_ERR_LIMIT;
    const size_t ybytes = sizeof(float) * static_cast<size_t>(s.out_elems());
    const size_t wtbytes = sizeof(float) * isc::repacked_filter_floats(sh.K, sh.C, sh.R, sh.S);
    if (overlap(y, ybytes, x, sizeof(float) * static_cast<size_t>(s.in_elems())) || overlap(y, ybytes, wt, wtbytes))
        return ISC_ERR_ALIAS;
    st = check_device();
    if (st) return st;
    isc::Decision dec{nullptr, 0, 0, isc::kGateAlways, nullptr};
    return hip_status(isc::launch_sparse_fused(sh, x, wt, y, dec, static_cast<hipStream_t>(stream)));
}

int isc_conv2d_dw_workspace_size(const isc_conv_desc *d, size_t *bytes) {
    if (!bytes) return ISC_ERR_NULL;
    Shape s;
    const int st = check_desc(d, &s);
    if (st) return st;
    const isc::SparseShape sh = sparse_shape(s);
    if (!isc::sparse_dw_applies(sh)) return ISC_ERR_LIMIT;
    *bytes = align_up(sizeof(float) * isc::sparse_dw_workspace_floats(sh), kAlign);
    return ISC_OK;
}

int isc_conv2d_dw(const isc_conv_desc *d, const float *x, const float *dy, float *dw, void *ws, size_t ws_bytes,
                  const isc_tuning *tuning, void *stream) {
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    if (!x || !dy || !dw || !ws) return ISC_ERR_NULL;
    if (!tuning_ok(tuning)) return ISC_ERR_ARG;
    if (!aligned(x, 4) || !aligned(dy, 4) || !aligned(dw, 4) || !aligned(ws, kAlign)) return ISC_ERR_ALIGN;
    const isc::SparseShape sh = sparse_shape(s, tuning);
    if (!isc::sparse_dw_applies(sh)) return ISC_ERR_LIMIT;
    const size_t need = align_up(sizeof(float) * isc::sparse_dw_workspace_floats(sh), kAlign);
    if (ws_bytes < need) return ISC_ERR_WORKSPACE;
    const size_t xb = sizeof(float) * static_cast<size_t>(s.in_elems());
    const size_t yb = sizeof(float) * static_cast<size_t>(s.out_elems());
    const size_t wb = sizeof(float) * static_cast<size_t>(s.filt_elems());
    if (overlap(dw, wb, x, xb) || overlap(dw, wb, dy, yb) || overlap(dw, wb, ws, need) || overlap(ws, need, x, xb) ||
        overlap(ws, need, dy, yb))
        return ISC_ERR_ALIAS;
    st = check_device();
    if (st) return st;
    return hip_status(isc::launch_sparse_dw(sh, x, dy, dw, static_cast<float *>(ws), static_cast<hipStream_t>(stream)));
}

int isc_sparse_kernel(const isc_conv_desc *d, int32_t *kernel) {
    if (!kernel) return ISC_ERR_NULL;
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    const isc::SparseShape sh = sparse_shape(s);
    const int fused = isc::sparse_fused_kernel(sh);
    *kernel = fused ? fused : isc::list_kernel_for(sh);
    return ISC_OK;
}

int isc_crossover_sparsity(const isc_conv_desc *d, double *sparsity) {
    if (!sparsity) return ISC_ERR_NULL;
    Shape s;
    const int st = check_desc(d, &s);
    if (st) return st;
    const isc::SparseShape sh = sparse_shape(s);
    const bool sparse_fits = isc::sparse_fused_applies(sh) || isc::sparse_conv_feasible(sh);
    const long long limit = sparse_fits ? isc::crossover_nnz_limit(sh) : -1;
    *sparsity = limit < 0 ? 2.0 : 1.0 - static_cast<double>(limit) / static_cast<double>(s.in_elems());
    return ISC_OK;
}

int isc_sparse_plan(const isc_conv_desc *d, const isc_tuning *tuning, isc_plan *plan) {
    if (!plan) return ISC_ERR_NULL;
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    if (!tuning_ok(tuning)) return ISC_ERR_ARG;
    const isc::SparseShape sh = sparse_shape(s, tuning);
    isc_plan p{};
    if (!isc::sparse_fused_plan_info(sh, &p)) {
        p = isc_plan{};
        p.kernel = isc::list_kernel_for(sh);
        p.waves = p.kernel == ISC_KERNEL_NONE ? 0 : isc::list_kernel_waves(p.kernel);
    }
    *plan = p;
    return ISC_OK;
}

int isc_read_decision(const void *ws, int32_t *path, uint64_t *nnz) {
    if (!ws || !path || !nnz) return ISC_ERR_NULL;
    const int st = check_device();
    if (st) return st;
    Ctrl c;
    if (hipMemcpy(&c, ws, sizeof(Ctrl), hipMemcpyDeviceToHost) != hipSuccess) return ISC_ERR_HIP;
    *path = static_cast<int32_t>(c.path_taken);
    *nnz = c.nnz_total;
    return ISC_OK;
}

int isc_decision(const isc_conv_desc *d, const void *ws, size_t ws_bytes, uint64_t *nnz_total,
                 int32_t *path_taken, void *stream) {
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    if (!ws || !nnz_total || !path_taken) return ISC_ERR_NULL;
    if (ws_bytes < sizeof(Ctrl)) return ISC_ERR_WORKSPACE;
    st = check_device();
    if (st) return st;
    Ctrl c;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    hipError_t e = hipMemcpyAsync(&c, ws, sizeof(Ctrl), hipMemcpyDeviceToHost, hs);
    if (e == hipSuccess) e = hipStreamSynchronize(hs);
    if (e != hipSuccess) return ISC_ERR_HIP;
    *nnz_total = c.nnz_total;
    *path_taken = static_cast<int32_t>(c.path_taken);
    return ISC_OK;
}

int isc_compact(const isc_conv_desc *d, const float *x, int32_t *row_ptr, isc_nz *nz,
                uint64_t *nnz_total, void *stream) {
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    if (!x || !row_ptr || !nz || !nnz_total) return ISC_ERR_NULL;
    if (!aligned(x, 4) || !aligned(row_ptr, 4) || !aligned(nz, 8) || !aligned(nnz_total, 8))
        return ISC_ERR_ALIGN;
    const size_t xb = sizeof(float) * static_cast<size_t>(s.in_elems());
    const size_t rb = sizeof(int32_t) * static_cast<size_t>(s.N * s.C * (s.H + 1));
    const size_t nb = sizeof(isc_nz) * static_cast<size_t>(s.in_elems());
    if (overlap(row_ptr, rb, x, xb) || overlap(nz, nb, x, xb) || overlap(nz, nb, row_ptr, rb) ||
        overlap(nnz_total, 8, x, xb) || overlap(nnz_total, 8, row_ptr, rb) || overlap(nnz_total, 8, nz, nb))
        return ISC_ERR_ALIAS;
    st = check_device();
    if (st) return st;
    static_assert(sizeof(isc_nz) == sizeof(NzEntry), "entry layout");
    static_assert(sizeof(unsigned long long) == sizeof(uint64_t), "counter layout");
    hipStream_t hs = static_cast<hipStream_t>(stream);
    unsigned long long *counter = reinterpret_cast<unsigned long long *>(nnz_total);
    hipError_t e = isc::launch_compact(x, static_cast<int>(s.N * s.C), static_cast<int>(s.H), static_cast<int>(s.W),
                                row_ptr, reinterpret_cast<NzEntry *>(nz), counter, hs);
    return hip_status(e);
}

int isc_repacked_filter_size(const isc_conv_desc *d, size_t *bytes) {
    if (!bytes) return ISC_ERR_NULL;
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    *bytes = sizeof(float) * isc::repacked_filter_floats(static_cast<int>(s.K), static_cast<int>(s.C),
                                                         static_cast<int>(s.R), static_cast<int>(s.S));
    return ISC_OK;
}

int isc_repack_filter(const isc_conv_desc *d, const float *w, float *wt, void *stream) {
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    if (!w || !wt) return ISC_ERR_NULL;
    if (!aligned(w, 4) || !aligned(wt, 16)) return ISC_ERR_ALIGN;
    const size_t wb = sizeof(float) * static_cast<size_t>(s.filt_elems());
    const size_t tb = sizeof(float) * isc::repacked_filter_floats(static_cast<int>(s.K), static_cast<int>(s.C),
                                                                  static_cast<int>(s.R), static_cast<int>(s.S));
    if (tb > static_cast<size_t>(kI32Max) * sizeof(float)) return ISC_ERR_LIMIT;
    if (overlap(w, wb, wt, tb)) return ISC_ERR_ALIAS;
    st = check_device();
    if (st) return st;
    return hip_status(isc::launch_repack_filter(w, static_cast<int>(s.K), static_cast<int>(s.C),
                                                static_cast<int>(s.R), static_cast<int>(s.S), wt,
                                                static_cast<hipStream_t>(stream)));
}

int isc_sparse_conv(const isc_conv_desc *d, const int32_t *row_ptr, const isc_nz *nz, const float *wt,
                    float *y, const isc_tuning *tuning, void *stream) {
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    if (!row_ptr || !nz || !wt || !y) return ISC_ERR_NULL;
    if (!tuning_ok(tuning)) return ISC_ERR_ARG;
    if (!aligned(row_ptr, 4) || !aligned(nz, 8) || !aligned(wt, 16) || !aligned(y, 4)) return ISC_ERR_ALIGN;
    const size_t yb = sizeof(float) * static_cast<size_t>(s.out_elems());
    const size_t tb = sizeof(float) * isc::repacked_filter_floats(static_cast<int>(s.K), static_cast<int>(s.C),
                                                                  static_cast<int>(s.R), static_cast<int>(s.S));
    if (overlap(y, yb, row_ptr, sizeof(int32_t) * static_cast<size_t>(s.N * s.C * (s.H + 1))) ||
        overlap(y, yb, nz, sizeof(isc_nz) * static_cast<size_t>(s.in_elems() + kNzTail)) ||
        overlap(y, yb, wt, tb))
        return ISC_ERR_ALIAS;
    const isc::SparseShape sh = sparse_shape(s, tuning);
    if (!isc::sparse_conv_feasible(sh)) return ISC_ERR_LIMIT;
    st = check_device();
    if (st) return st;
    isc::Decision dec{nullptr, 0, 0, isc::kGateAlways, nullptr};
    return hip_status(isc::launch_sparse_conv(sh, row_ptr, reinterpret_cast<const NzEntry *>(nz), wt, y, dec,
                                              static_cast<hipStream_t>(stream)));
}

int isc_im2col(const isc_conv_desc *d, const float *x, float *col, int64_t ldc, void *stream) {
    Shape s;
    int st = check_desc(d, &s);
    if (st) return st;
    if (!x || !col) return ISC_ERR_NULL;
    if (ldc < s.ncols() || s.crs() * ldc > kI32Max) return ISC_ERR_ARG;
    if (!aligned(x, 4) || !aligned(col, 4)) return ISC_ERR_ALIGN;
    if (overlap(col, sizeof(float) * static_cast<size_t>(s.crs() * ldc), x,
                sizeof(float) * static_cast<size_t>(s.in_elems())))
        return ISC_ERR_ALIAS;
    st = check_device();
    if (st) return st;
    isc::Decision dec{nullptr, 0, 0, isc::kGateAlways, nullptr};
    return hip_status(isc::launch_im2col(x, static_cast<int>(s.N), static_cast<int>(s.C), static_cast<int>(s.H),
                                         static_cast<int>(s.W), static_cast<int>(s.R), static_cast<int>(s.S),
                                         static_cast<int>(s.T), static_cast<int>(s.P), static_cast<int>(s.Ho),
                                         static_cast<int>(s.Wo), col, ldc, dec,
                                         static_cast<hipStream_t>(stream)));
}

int isc_gemm_f32(int32_t M, int32_t Ncols, int32_t Kd, const float *a, int64_t lda, const float *b,
                 int64_t ldb, float *c, int64_t ldc, void *stream) {
    if (M < 1 || Ncols < 1 || Kd < 1) return ISC_ERR_SHAPE;
    if (!a || !b || !c) return ISC_ERR_NULL;
    if (lda < Kd || ldb < Ncols || ldc < Ncols) return ISC_ERR_SHAPE;
    if (static_cast<int64_t>(M) * lda > kI32Max || static_cast<int64_t>(Kd) * ldb > kI32Max ||
        static_cast<int64_t>(M) * ldc > kI32Max || (M + 31) / 32 > 65535)
        return ISC_ERR_LIMIT;
    if (!aligned(a, 4) || !aligned(b, 4) || !aligned(c, 4)) return ISC_ERR_ALIGN;
    const size_t cb = sizeof(float) * static_cast<size_t>((M - 1) * ldc + Ncols);
    if (overlap(c, cb, a, sizeof(float) * static_cast<size_t>((M - 1) * lda + Kd)) ||
        overlap(c, cb, b, sizeof(float) * static_cast<size_t>((Kd - 1) * ldb + Ncols)))
        return ISC_ERR_ALIAS;
    int st = check_device();
    if (st) return st;
    isc::Decision dec{nullptr, 0, 0, isc::kGateAlways, nullptr};
    return hip_status(isc::launch_gemm_f32(M, Ncols, Kd, a, lda, b, ldb, c, ldc, 0, false, dec,
                                           static_cast<hipStream_t>(stream)));
}

}  // extern "C"
