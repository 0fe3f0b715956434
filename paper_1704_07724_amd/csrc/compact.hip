// ISC step 1 (Sec. "Sparse Convolution"): turn every (n, c) input plane into
// a row-major list of its nonzero values with their row and column, plus
// per-row offsets, using wavefront ballots and in-wave prefix counts.
//
// One wavefront owns one plane at a time.  It reads the plane in 64-element
// chunks (kUnroll chunks in flight per lane), takes a 64-bit ballot of the
// nonzero predicate, and gives every nonzero lane its output slot with
// mbcnt (the number of set ballot bits below the lane).  The lane holding
// the first element of a row writes that row's offset.  The per-plane lists
// are dense in fixed H*W slots, so the output is unique and needs no second
// pass.  Traffic: 4 bytes read per input element, 8 bytes written per
// nonzero, 4 bytes per row offset.  A second, one-workgroup kernel adds the
// per-plane counts into the total the dispatcher reads.
#include "isc_internal.hpp"

namespace isc {
namespace {

constexpr int kWaves = 4;    // wavefronts per workgroup
constexpr int kUnroll = 8;   // 64-element chunks loaded before the ballots

__device__ __forceinline__ uint32_t lanes_below(unsigned long long mask) {
    return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

__global__ __launch_bounds__(kWaves * 64)
void compact_kernel(const float *__restrict__ x, int planes, int H, int W,
                    int32_t *__restrict__ row_ptr, NzEntry *__restrict__ nz) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int HW = H * W;
    // (row, column) of this lane's element in the first chunk, and the step
    // that moves it 64 elements further in row-major order
    const int y_first = lane / W;
    const int x_first = lane - y_first * W;
    const int dy = 64 / W;
    const int dx = 64 - dy * W;

    for (int p = blockIdx.x * kWaves + wave; p < planes; p += gridDim.x * kWaves) {
        const float *xp = x + static_cast<size_t>(p) * HW;
        NzEntry *np = nz + static_cast<size_t>(p) * HW;
        int32_t *rp = row_ptr + static_cast<size_t>(p) * (H + 1);
        uint32_t base = 0;  // nonzeros before the current chunk (wave-uniform)
        int y = y_first, xc = x_first;
        for (int e0 = 0; e0 < HW; e0 += 64 * kUnroll) {
            float v[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int e = e0 + u * 64 + lane;
                v[u] = e < HW ? xp[e] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int e = e0 + u * 64 + lane;
                const bool inside = e < HW;
                const uint32_t bits = __float_as_uint(v[u]);
                const bool nonzero = inside && (bits & 0x7fffffffu) != 0u;
                const unsigned long long mask = __ballot(nonzero);
                const uint32_t slot = base + lanes_below(mask);
                if (nonzero) {
                    NzEntry ent;
                    ent.v = v[u];
                    ent.yx = (static_cast<uint32_t>(y) << 16) | static_cast<uint32_t>(xc);
                    np[slot] = ent;
                }
                if (inside && xc == 0) rp[y] = static_cast<int32_t>(slot);
                base += static_cast<uint32_t>(__popcll(mask));
                xc += dx;
                y += dy;
                if (xc >= W) {
                    xc -= W;
                    ++y;
                }
            }
        }
        if (lane == 0) rp[H] = static_cast<int32_t>(base);
    }
}

// Total of the per-plane counts (row_ptr[p][H]) by one workgroup, written
// to *total with a plain store: no counter to clear, no same-address atomics.
constexpr int kCountThreads = 1024;

__global__ __launch_bounds__(kCountThreads)
void count_kernel(const int32_t *__restrict__ row_ptr, int planes, int H,
                  unsigned long long *__restrict__ total) {
    __shared__ unsigned long long part[kCountThreads / 64];
    unsigned long long s = 0;
    for (int p = threadIdx.x; p < planes; p += kCountThreads)
        s += static_cast<uint32_t>(row_ptr[static_cast<size_t>(p) * (H + 1) + H]);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long t = 0;
#pragma unroll
        for (int i = 0; i < kCountThreads / 64; ++i) t += part[i];
        *total = t;
    }
}

}  // namespace

hipError_t launch_compact(const float *x, int planes, int H, int W, int32_t *row_ptr,
                          NzEntry *nz, unsigned long long *counter, hipStream_t s) {
    // one wavefront per plane; enough workgroups to cover 256 CUs many times
    int groups = (planes + kWaves - 1) / kWaves;
    if (groups > 8192) groups = 8192;
    compact_kernel<<<groups, kWaves * 64, 0, s>>>(x, planes, H, W, row_ptr, nz);
    count_kernel<<<1, kCountThreads, 0, s>>>(row_ptr, planes, H, counter);
    return hipGetLastError();
}

}  // namespace isc
