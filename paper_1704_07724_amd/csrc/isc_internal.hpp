// Internal declarations shared by the library's translation units (not part
// of the C ABI; include/isc.h is).
#pragma once

#include <hip/hip_runtime.h>
#include "isc.h"
#include <cstddef>
#include <cstdint>

namespace isc {

// Device image of isc_nz: value bits and (row << 16) | column.
struct alignas(8) NzEntry {
    float v;
    uint32_t yx;
};

// Control block at offset 0 of every workspace.
struct alignas(16) Ctrl {
    unsigned long long nnz_total;  // nonzero inputs counted by the compaction
    uint32_t path_taken;           // 1 = sparse, 2 = dense (isc_path values)
    uint32_t sink;                 // written (rarely) by cache warm-ups, never read
};

// Whether a kernel of one path runs unconditionally or only when the
// device-side decision picks its path.
enum Gate : int { kGateAlways = 0, kGateIfSparse = 1, kGateIfDense = 2 };

// Per-workgroup nonzero counts written by the compaction, at most this many
// (a multiple of 4; unused entries are zero).
constexpr int kMaxParts = 1024;

// Census of a layer's output: its nonzero count, kept as one count per
// workgroup of the kernel that wrote the output (so no counter needs
// clearing and no atomics are involved).  The next layer's decision sums the
// counts instead of reading its input again.  Header, then the counts.
struct alignas(16) CensusHeader {
    unsigned long long elems;  // entries of the output the counts cover
    uint32_t nslots;           // counts in use, a multiple of 4 (zero tail)
    uint32_t reserved;
};

// Output epilogue of the kernels that write y: the rectifier of Eq. 2 and
// the census of the rectified output.
struct Epilogue {
    int relu;                  // store max(0, v) (v > 0 ? v : +0, NaN -> +0)
    CensusHeader *census;      // nullptr: no census
    uint32_t cap;              // counts the census has room for
    unsigned long long elems;  // entries of y
};

// Device-side decision: sparse iff the input's nonzero count, the sum of the
// compaction's per-workgroup counts (or of a census of the input), is <=
// nnz_limit.  A kernel launched after the one that recorded the decision
// reads the recorded path instead.
struct Decision {
    const uint32_t *parts;         // per-workgroup counts (nullptr: no compaction ran)
    int nparts;                    // entries of parts, a multiple of 4
    long long nnz_limit;           // largest nonzero count that still picks sparse (-1: none does)
    int gate;
    Ctrl *record;                  // where block 0 records count and path (may be nullptr)
    const Ctrl *recorded = nullptr;  // decision recorded by an earlier kernel on the stream
};

// Sum of n counts (n a multiple of 4), by the calling wavefront (every lane
// gets the total).
__device__ __forceinline__ unsigned long long sum_counts(const uint32_t *counts, int n) {
    unsigned long long s = 0;
    const uint4 *p = reinterpret_cast<const uint4 *>(counts);
    const int n4 = n / 4;
    const int lane = threadIdx.x & 63;
    if (n4 <= 64) {  // one load per lane at most
        if (lane < n4) {
            const uint4 v = p[lane];
            s = static_cast<unsigned long long>(v.x) + v.y + v.z + v.w;
        }
    } else {
        // eight loads in flight per lane (a census of thousands of slots would
        // otherwise cost one dependent L2 round trip per 64 of them, in every
        // wavefront's prologue); indices past the end load the last word again
        // and are not added
        for (int base = lane; base < n4; base += 8 * 64) {
            uint4 v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = p[min(base + j * 64, n4 - 1)];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (base + j * 64 < n4) s += static_cast<unsigned long long>(v[j].x) + v[j].y + v[j].z + v[j].w;
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    return s;
}

// The input's nonzero count for the decision, by the calling wavefront;
// all ones when no count ran or the parts say "unknown" (a sum of 2^32 or
// more: the census reduction's mark of an unusable census, as real counts
// are below 2^31).
__device__ __forceinline__ unsigned long long decision_total(const Decision &d) {
    if (!d.parts) return ~0ull;
    const unsigned long long s = sum_counts(d.parts, d.nparts);
    return s >= (1ull << 32) ? ~0ull : s;
}

// Gate of a kernel on path `mine` (1 sparse, 2 dense): whether it runs.
// Block 0 records the count (all ones when no count is known) and the path
// taken when asked.  Called by whole wavefronts.
__device__ __forceinline__ bool decision_gate(const Decision &d, uint32_t mine) {
    if (d.recorded) return d.recorded->path_taken == mine;
    const bool recorder = d.record && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0;
    if (d.gate == kGateAlways && !recorder) return true;  // no count needed
    const unsigned long long total = decision_total(d);
    const bool sparse = total != ~0ull && static_cast<long long>(total) <= d.nnz_limit;
    const bool run = d.gate == kGateAlways || (d.gate == kGateIfSparse ? sparse : !sparse);
    if (d.record && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && threadIdx.x == 0) {
        d.record->nnz_total = total;
        d.record->path_taken = run ? mine : 3u - mine;
    }
    return run;
}

// The stored value under the epilogue: the rectifier when asked.
__device__ __forceinline__ float epilogue_value(float v, int relu) { return relu && !(v > 0.0f) ? 0.0f : v; }

// 1 if the stored value is nonzero (the compaction's zero test: +0 and -0
// are zero).
__device__ __forceinline__ uint32_t nonzero_bit(float v) { return (__float_as_uint(v) & 0x7fffffffu) != 0u; }

// The workgroup's census count: the sum of every thread's `cnt` into the
// workgroup's slot; block 0 also writes the header and clears the tail
// slots up to a multiple of 4.  Called by every thread of the workgroup
// (uniformly: it synchronises); `sums` is LDS with one word per wavefront,
// `stride` words apart, that nothing else touches until the call returns.
__device__ __forceinline__ void census_commit(const Epilogue &e, uint32_t cnt, uint32_t *sums, int stride = 1) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) sums[wave * stride] = cnt;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
        for (int i = 0; i < static_cast<int>(blockDim.x >> 6); ++i) t += sums[i * stride];
        const uint32_t nblocks = gridDim.x * gridDim.y * gridDim.z;
        const uint32_t b = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
        uint32_t *slots = reinterpret_cast<uint32_t *>(e.census + 1);
        slots[b] = t;
        if (b == 0) {
            const uint32_t n4 = (nblocks + 3u) & ~3u;
            for (uint32_t i = nblocks; i < n4; ++i) slots[i] = 0u;
            CensusHeader h;
            h.elems = e.elems;
            h.nslots = n4;
            h.reserved = 0u;
            *e.census = h;
        }
    }
}

// Census slots a launch of `blocks` workgroups needs.
inline uint32_t census_slots_for(int64_t blocks) { return static_cast<uint32_t>((blocks + 3) / 4 * 4); }

// --- launchers (each returns hipGetLastError() of its launches) ------------

// ISC step 1: per-plane row-major nonzero lists, then their total in *counter.
hipError_t launch_compact(const float *x, int planes, int H, int W, int32_t *row_ptr,
                          NzEntry *nz, unsigned long long *counter, hipStream_t s);

// A census's total into parts[0 .. 4) (the decision's input for a layer
// whose input carries a census): one workgroup sums the census's counts; a
// census that does not cover exactly `elems` entries, or claims more counts
// than `cap`, leaves all ones (a sum the decision reads as "unknown").
// The same launch also reads `warm_bytes` bytes at `warm` (a filter the
// next kernel streams in small dependent steps) with its other workgroups,
// so that the kernel finds them in the last-level cache instead of HBM.
hipError_t launch_census_parts(const CensusHeader *census, uint32_t cap, unsigned long long elems, uint32_t *parts,
                               const void *warm, size_t warm_bytes, Ctrl *ctrl, hipStream_t s);

// Nonzero count of x[0 .. total) as per-workgroup parts (the decision's input
// when the sparse path compacts on the fly); with w, extra workgroups of the
// same launch repack the K x C x R x S filter into wt (layout of
// launch_repack_filter); without w, extra workgroups warm the cache with
// warm_bytes bytes at `warm` (as launch_census_parts does).
hipError_t launch_count_parts(const float *x, int64_t total, uint32_t *parts, int *nparts, hipStream_t s,
                              const float *w = nullptr, int K = 0, int C = 0, int R = 0, int S = 0,
                              float *wt = nullptr, const void *warm = nullptr, size_t warm_bytes = 0,
                              Ctrl *ctrl = nullptr);

// The sparse path's first kernel: ISC step 1 with per-workgroup counts in
// parts (kMaxParts entries; *nparts gets the number in use), and the filter
// repack into wt in the same launch.
hipError_t launch_prep(const float *x, int planes, int H, int W, int32_t *row_ptr, NzEntry *nz,
                       uint32_t *parts, int *nparts, const float *w, int K, int C, int R, int S,
                       float *wt, hipStream_t s);

// Filter repack KCRS -> ISC step 2's K-contiguous layout:
// wt[((c*R + r)*S + s)*Kp + k], Kp = K rounded up to 64, zero padded.
size_t repacked_filter_floats(int K, int C, int R, int S);
hipError_t launch_repack_filter(const float *w, int K, int C, int R, int S, float *wt, hipStream_t s);

struct SparseShape {
    int N, C, H, W, K, R, S, T, P, Ho, Wo;
    isc_tuning tu;  // the caller's plan overrides (all zero: the library chooses)
};

// ISC steps 1-3 in one launch, compacting on the fly from x, with the filter
// repacked K-contiguous (launch_repack_filter's layout; square 1x1/3x3/5x5
// filters at stride 1, 3x3/5x5 at stride 2 with at most 8 output columns).
// The filter-resident kernel takes filters that fit in LDS (K <= 64; with
// the weights streamed to registers when no two wavefronts share a
// channel); the filter-ring kernel (sparse_fring.hip) streams larger ones
// through LDS (stride 1).
bool sparse_fused_applies(const SparseShape &sh);
hipError_t launch_sparse_fused(const SparseShape &sh, const float *x, const float *wt, float *y, const Decision &dec,
                               hipStream_t s, const Epilogue &epi = Epilogue{});
bool sparse_fring_applies(const SparseShape &sh);
// 1 (filter-resident), 6 (filter-resident plan with the weights streamed to
// registers), 5 (filter-ring) or 0 (none): isc_sparse_kernel's ids.
int sparse_fused_kernel(const SparseShape &sh);
hipError_t launch_sparse_fring(const SparseShape &sh, const float *x, const float *wt, float *y, const Decision &dec,
                               hipStream_t s, const Epilogue &epi = Epilogue{});
// The plan the on-the-fly kernels take for a shape (false: none takes it).
bool sparse_fused_plan_info(const SparseShape &sh, isc_plan *out);
bool sparse_fring_plan_info(const SparseShape &sh, isc_plan *out);
int64_t sparse_fring_max_groups(const SparseShape &sh);
// Upper bound of the workgroups of the on-the-fly kernels' launch for a
// shape (the census slots their epilogue may write).
int64_t sparse_fused_max_groups(const SparseShape &sh);

// Weight gradient of Eq. 1 from the nonzero inputs (stride 1, square 1x1,
// 3x3 or 5x5 filters): per-range sums into part (sparse_dw_workspace_floats
// floats), then their ordered sum into dw (K x C x R x S).
bool sparse_dw_applies(const SparseShape &sh);
size_t sparse_dw_workspace_floats(const SparseShape &sh);
hipError_t launch_sparse_dw(const SparseShape &sh, const float *x, const float *dy, float *dw, float *part,
                            hipStream_t s);

// Which kernel runs over compacted lists for a shape (the values are those
// of isc_sparse_kernel in the C ABI).
enum ListKernel : int { kListNone = 0, kListResident = 2, kListRing = 3, kListGeneric = 4 };
int list_kernel_for(const SparseShape &sh);
// Wavefronts per workgroup of a list kernel.
int list_kernel_waves(int kernel);

// AUTO's per-shape crossover: the largest nonzero count of the input at
// which the sparse path is expected to be faster than the dense path for
// this shape, -1 when it never is (crossover.hip).
long long crossover_nnz_limit(const SparseShape &sh);
// The dense path's expected time (ms) for an M x Ncols x Kd implicit GEMM,
// from its tile grid (dense_conv.hip).
double dense_time_model(int64_t M, int64_t Ncols, int64_t Kd);

// ISC steps 2 and 3: zero-skipping convolution over the compacted lists.
hipError_t launch_sparse_conv(const SparseShape &sh, const int32_t *row_ptr,
                              const NzEntry *nz, const float *wt, float *y,
                              const Decision &dec, hipStream_t s);

// Dense baseline of Fig. 3: im2col then the fp32 MFMA GEMM.
hipError_t launch_im2col(const float *x, int N, int C, int H, int W, int R, int S,
                         int T, int P, int Ho, int Wo, float *col, int64_t ldc,
                         const Decision &dec, hipStream_t s);

// c = a * b, row-major; when conv_hw > 0 the output column n is scattered to
// y[((n / conv_hw) * M + m) * conv_hw + n % conv_hw] (NCHW) instead of
// c[m * ldc + n].  b_padded: every row of b is readable up to a multiple of
// 256 columns (true for the library's own im2col buffer).
hipError_t launch_gemm_f32(int M, int Ncols, int Kd, const float *a, int64_t lda,
                           const float *b, int64_t ldb, float *c, int64_t ldc,
                           int conv_hw, bool b_padded, const Decision &dec,
                           hipStream_t s, const Epilogue &epi = Epilogue{});

// The dense baseline as one implicit GEMM: the fp32 MFMA GEMM of Fig. 3 with
// the im2col matrix gathered from x while loading (C*R*S < 2^16), output
// scattered to NCHW.
bool conv_gemm_implicit_ok(int C, int R, int S);
// part: the partial sums of a split reduction (conv_gemm_split_floats
// floats), or nullptr for one range.
hipError_t launch_conv_gemm(const float *x, const float *w, float *y, int N, int C, int H, int W, int K, int R,
                            int S, int T, int P, int Ho, int Wo, const Decision &dec, hipStream_t s,
                            const Epilogue &epi = Epilogue{}, float *part = nullptr);
// Floats of the partial sums launch_conv_gemm splits its reduction into for
// an M x Ncols x Kd product, 0 when it does not split (grids that fill the
// chip, or short reductions).
size_t conv_gemm_split_floats(int M, int64_t Ncols, int Kd);
// Upper bound of the GEMM's workgroups for an M x Ncols product (the census
// slots its epilogue may write).
int64_t gemm_max_groups(int64_t M, int64_t Ncols);

// The epilogue as a pass of its own over y[0 .. n) (in place), for the
// kernels that have none: at most kRectifyGroups workgroups.
constexpr int kRectifyGroups = 1024;
hipError_t launch_rectify(float *y, int64_t n, const Epilogue &epi, const Decision &dec, hipStream_t s);

}  // namespace isc
