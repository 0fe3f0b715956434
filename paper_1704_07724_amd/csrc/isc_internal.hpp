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

// Device-side decision: sparse iff nnz <= nnz_limit.
struct Decision {
    const Ctrl *ctrl;             // nnz_total source (unused when gate == Always)
    unsigned long long nnz_limit; // largest nonzero count that still picks sparse
    int gate;
    Ctrl *record;                 // where block 0 records the path taken (may be nullptr)
};

__device__ __forceinline__ bool decision_says_run(const Decision &d) {
    if (d.gate == kGateAlways) return true;
    const bool sparse = d.ctrl->nnz_total <= d.nnz_limit;
    return d.gate == kGateIfSparse ? sparse : !sparse;
}

// --- launchers (each returns hipGetLastError() of its launches) ------------

// ISC step 1: per-plane row-major nonzero lists, then their total in *counter.
hipError_t launch_compact(const float *x, int planes, int H, int W, int32_t *row_ptr,
                          NzEntry *nz, unsigned long long *counter, hipStream_t s);

// Filter repack KCRS -> ISC step 2's K-contiguous kernel matrix, blocked by
// 64 output maps: wt[((c*ceil(K/64) + kb)*64 + l)*RSP + t], RSP = R*S
// rounded up to 4, zero padded.
size_t repacked_filter_floats(int K, int C, int R, int S);
hipError_t launch_repack_filter(const float *w, int K, int C, int R, int S, float *wt, hipStream_t s);

struct SparseShape {
    int N, C, H, W, K, R, S, T, P, Ho, Wo;
};

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

}  // namespace isc
