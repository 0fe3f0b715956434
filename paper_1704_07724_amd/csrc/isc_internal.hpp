// Internal declarations shared by the library's translation units (not part
// of the C ABI; include/isc.h is).
#pragma once

#include <hip/hip_runtime.h>
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
    uint32_t reserved;
};

// Whether a kernel of one path runs unconditionally or only when the
// device-side decision picks its path.
enum Gate : int { kGateAlways = 0, kGateIfSparse = 1, kGateIfDense = 2 };

// Per-workgroup nonzero counts written by the compaction, at most this many
// (a multiple of 4; unused entries are zero).
constexpr int kMaxParts = 1024;

// Device-side decision: sparse iff the input's nonzero count, the sum of the
// compaction's per-workgroup counts, is <= nnz_limit.  A kernel launched
// after the one that recorded the decision reads the recorded path instead.
struct Decision {
    const uint32_t *parts;         // per-workgroup counts (nullptr: no compaction ran)
    int nparts;                    // entries of parts, a multiple of 4
    unsigned long long nnz_limit;  // largest nonzero count that still picks sparse
    int gate;
    Ctrl *record;                  // where block 0 records count and path (may be nullptr)
    const Ctrl *recorded = nullptr;  // decision recorded by an earlier kernel on the stream
};

// Sum of the per-workgroup counts, by the calling wavefront (every lane gets
// the total).
__device__ __forceinline__ unsigned long long decision_total(const Decision &d) {
    unsigned long long s = 0;
    const uint4 *p = reinterpret_cast<const uint4 *>(d.parts);
    for (int i = threadIdx.x & 63; i < d.nparts / 4; i += 64) {
        const uint4 v = p[i];
        s += static_cast<unsigned long long>(v.x) + v.y + v.z + v.w;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    return s;
}

// Gate of a kernel on path `mine` (1 sparse, 2 dense): whether it runs.
// Block 0 records the count (all ones when no compaction ran) and the path
// taken when asked.  Called by whole wavefronts.
__device__ __forceinline__ bool decision_gate(const Decision &d, uint32_t mine) {
    if (d.recorded) return d.recorded->path_taken == mine;
    const unsigned long long total = d.parts ? decision_total(d) : ~0ull;
    const bool sparse = d.parts != nullptr && total <= d.nnz_limit;
    const bool run = d.gate == kGateAlways || (d.gate == kGateIfSparse ? sparse : !sparse);
    if (d.record && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) {
        d.record->nnz_total = total;
        d.record->path_taken = run ? mine : 3u - mine;
    }
    return run;
}

// --- launchers (each returns hipGetLastError() of its launches) ------------

// ISC step 1: per-plane row-major nonzero lists, then their total in *counter.
hipError_t launch_compact(const float *x, int planes, int H, int W, int32_t *row_ptr,
                          NzEntry *nz, unsigned long long *counter, hipStream_t s);

// Nonzero count of x[0 .. total) as per-workgroup parts (the decision's input
// when the sparse path compacts on the fly); with w, extra workgroups of the
// same launch repack the K x C x R x S filter into wt (layout of
// launch_repack_filter).
hipError_t launch_count_parts(const float *x, int64_t total, uint32_t *parts, int *nparts, hipStream_t s,
                              const float *w = nullptr, int K = 0, int C = 0, int R = 0, int S = 0,
                              float *wt = nullptr);

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
};

// ISC steps 1-3 in one launch, compacting on the fly from x, with the filter
// repacked K-contiguous (launch_repack_filter's layout; stride 1, square
// 1x1/3x3/5x5 filters).
// The filter-resident kernel takes filters that fit in LDS (K <= 64); the
// filter-ring kernel (sparse_fring.hip) streams larger ones through LDS.
bool sparse_fused_applies(const SparseShape &sh);
hipError_t launch_sparse_fused(const SparseShape &sh, const float *x, const float *wt, float *y, const Decision &dec,
                               hipStream_t s);
bool sparse_fring_applies(const SparseShape &sh);
// 1 (filter-resident), 5 (filter-ring) or 0 (neither): isc_sparse_kernel's ids.
int sparse_fused_kernel(const SparseShape &sh);
hipError_t launch_sparse_fring(const SparseShape &sh, const float *x, const float *wt, float *y, const Decision &dec,
                               hipStream_t s);

// Which kernel runs over compacted lists for a shape (the values are those
// of isc_sparse_kernel in the C ABI).
enum ListKernel : int { kListNone = 0, kListResident = 2, kListRing = 3, kListGeneric = 4 };
int list_kernel_for(const SparseShape &sh);

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
                           hipStream_t s);

// The dense baseline as one implicit GEMM: the fp32 MFMA GEMM of Fig. 3 with
// the im2col matrix gathered from x while loading (C*R*S < 2^16), output
// scattered to NCHW.
bool conv_gemm_implicit_ok(int C, int R, int S);
hipError_t launch_conv_gemm(const float *x, const float *w, float *y, int N, int C, int H, int W, int K, int R,
                            int S, int T, int P, int Ho, int Wo, const Decision &dec, hipStream_t s);

}  // namespace isc
