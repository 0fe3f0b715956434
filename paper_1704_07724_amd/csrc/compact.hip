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
// nonzero, 4 bytes per row offset.
//
// The sparse path runs the compaction inside one "prep" launch together with
// the filter repack (ISC step 2's K-contiguous layout: extra workgroups each
// transpose a 64 x 64 tile), and each compaction workgroup stores its own
// nonzero count; the kernels after it add those counts for the sparse/dense
// decision.  The stand-alone entry point instead sums the per-plane counts
// in a second launch spread over the CUs, one atomic add per workgroup.
#include "isc_internal.hpp"

#include <algorithm>

namespace isc {
namespace {

constexpr int kWaves = 4;    // wavefronts per workgroup
constexpr int kUnroll = 16;  // 64-element chunks loaded before the ballots (a 32 x 32 plane at once)

// Loads of data read once (the input's zero test): the non-temporal cache
// policy.  Measured on a cold 36 MB input behind 512 MiB of dirty cache
// lines, it halves the read time against the default policy, which
// allocates the lines in L2 at the cost of evicting dirty ones.
typedef float float4_nt __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float load_once(const float *p) { return __builtin_nontemporal_load(p); }

__device__ __forceinline__ float4 load_once(const float4 *p) {
    const float4_nt v = __builtin_nontemporal_load(reinterpret_cast<const float4_nt *>(p));
    return make_float4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ uint32_t lanes_below(unsigned long long mask) {
    return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

// Compact planes p = first, first + stride, ... (< planes) with the calling
// wavefront; returns the number of nonzeros it listed (wave-uniform).
//
// Planes of at most kBatch elements (every workload layer's) take one batch
// of kUnroll chunks each.  A lane's positions in the chunks are then the
// same in every plane: the wavefront computes them once (packed row and
// column, and which chunks start a row at the lane), so that listing a chunk
// is the zero test, the ballot, the lane's slot (mbcnt), the entry store
// and, at row starts, the row offset store.  The next plane's loads are
// issued before the current plane is listed.  Larger planes take several
// batches, with the positions stepped along.
constexpr int kBatch = 64 * kUnroll;

__device__ __forceinline__ uint32_t compact_planes(const float *__restrict__ x, int planes, int H, int W,
                                                   int32_t *__restrict__ row_ptr, NzEntry *__restrict__ nz,
                                                   int first, int stride) {
    const int lane = threadIdx.x & 63;
    const int HW = H * W;
    uint32_t listed = 0;
    if (first >= planes) return 0;

    auto load_batch = [&](int p, int e0, float (&v)[kUnroll]) {
        const float *xp = x + static_cast<size_t>(p) * HW;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int e = e0 + u * 64 + lane;
            v[u] = e < HW ? load_once(xp + e) : 0.0f;  // past the plane: zero, never listed
        }
    };

    if (HW <= kBatch) {
        uint32_t yx[kUnroll];
        uint32_t row_start = 0;  // bit u: the lane holds a row's first element in chunk u
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int e = u * 64 + lane;
            const int yy = e / W, xx = e - (e / W) * W;
            yx[u] = (static_cast<uint32_t>(yy) << 16) | static_cast<uint32_t>(xx);
            row_start |= static_cast<uint32_t>(e < HW && xx == 0) << u;
        }
        float cur[kUnroll];
        load_batch(first, 0, cur);
        for (int p = first; p < planes; p += stride) {
            float nxt[kUnroll];
            if (p + stride < planes) load_batch(p + stride, 0, nxt);
            NzEntry *np = nz + static_cast<size_t>(p) * HW;
            int32_t *rp = row_ptr + static_cast<size_t>(p) * (H + 1);
            uint32_t base = 0;  // nonzeros of the plane before the current chunk (wave-uniform)
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const bool nonzero = (__float_as_uint(cur[u]) & 0x7fffffffu) != 0u;
                const unsigned long long mask = __ballot(nonzero);
                const uint32_t slot = base + lanes_below(mask);
                if (nonzero) {
                    NzEntry ent;
                    ent.v = cur[u];
                    ent.yx = yx[u];
                    np[slot] = ent;
                }
                if (row_start & (1u << u)) rp[yx[u] >> 16] = static_cast<int32_t>(slot);
                base += static_cast<uint32_t>(__popcll(mask));
            }
            if (lane == 0) rp[H] = static_cast<int32_t>(base);
            listed += base;
            __builtin_memcpy(cur, nxt, sizeof(cur));
        }
        return listed;
    }

    // (row, column) of this lane's element in a plane's first chunk, and the
    // step that moves it 64 elements further in row-major order
    const int y_first = lane / W;
    const int x_first = lane - y_first * W;
    const int dy = 64 / W;
    const int dx = 64 - dy * W;
    int p = first, e0 = 0;
    float cur[kUnroll];
    load_batch(p, e0, cur);
    uint32_t base = 0;
    int y = y_first, xc = x_first;
    for (;;) {
        // the batch after this one: the next kBatch elements of this plane,
        // else the first of the wavefront's next plane
        int pn = p, en = e0 + kBatch;
        if (en >= HW) {
            en = 0;
            pn = p + stride;
        }
        float nxt[kUnroll];
        if (pn < planes) load_batch(pn, en, nxt);

        NzEntry *np = nz + static_cast<size_t>(p) * HW;
        int32_t *rp = row_ptr + static_cast<size_t>(p) * (H + 1);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int e = e0 + u * 64 + lane;
            const bool inside = e < HW;
            const bool nonzero = (__float_as_uint(cur[u]) & 0x7fffffffu) != 0u;
            const unsigned long long mask = __ballot(nonzero);
            const uint32_t slot = base + lanes_below(mask);
            if (nonzero) {
                NzEntry ent;
                ent.v = cur[u];
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
        if (pn != p) {  // the plane is done: its count, and a fresh walk
            if (lane == 0) rp[H] = static_cast<int32_t>(base);
            listed += base;
            base = 0;
            y = y_first;
            xc = x_first;
        }
        if (pn >= planes) break;
        p = pn;
        e0 = en;
        __builtin_memcpy(cur, nxt, sizeof(cur));
    }
    return listed;
}

// The stand-alone compaction; workgroup 0 also clears the total, which the
// count kernel after it accumulates.
__global__ __launch_bounds__(kWaves * 64)
void compact_kernel(const float *__restrict__ x, int planes, int H, int W,
                    int32_t *__restrict__ row_ptr, NzEntry *__restrict__ nz, unsigned long long *__restrict__ total) {
    if (blockIdx.x == 0 && threadIdx.x == 0) *total = 0ull;
    const int wave = threadIdx.x >> 6;
    compact_planes(x, planes, H, W, row_ptr, nz, blockIdx.x * kWaves + wave, gridDim.x * kWaves);
}

// Total of the per-plane counts (row_ptr[p][H], H + 1 words apart): one
// plane per thread over as many workgroups as it takes (every count in one
// round trip, spread over the CUs), each workgroup adding its sum to *total
// with one atomic (a few dozen atomics on one address in all).
constexpr int kCountThreads = 256;

__global__ __launch_bounds__(kCountThreads)
void count_kernel(const int32_t *__restrict__ row_ptr, int planes, int H,
                  unsigned long long *__restrict__ total) {
    __shared__ unsigned long long part[kCountThreads / 64];
    const int p = blockIdx.x * kCountThreads + static_cast<int>(threadIdx.x);
    unsigned long long s = p < planes ? static_cast<uint32_t>(row_ptr[static_cast<size_t>(p) * (H + 1) + H]) : 0u;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long t = 0;
#pragma unroll
        for (int i = 0; i < kCountThreads / 64; ++i) t += part[i];
        atomicAdd(total, t);
    }
}

// One 64 x 64 tile of the filter repack through LDS: reads along q = (c, r,
// s), writes along k:  wt[q * Kp + k] = w[k * CRS + q]  (0 for k >= K).
__device__ __forceinline__ void repack_tile(const float *__restrict__ w, int K, int Kp, int CRS,
                                            float *__restrict__ wt, int qt, int kt, float (&tile)[64][65]) {
    const int q0 = qt * 64, k0 = kt * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const int waves = static_cast<int>(blockDim.x >> 6);
    for (int i = ty; i < 64; i += waves) {
        const int k = k0 + i, q = q0 + tx;
        tile[i][tx] = (k < K && q < CRS) ? w[static_cast<size_t>(k) * CRS + q] : 0.0f;
    }
    __syncthreads();
    for (int i = ty; i < 64; i += waves) {
        const int q = q0 + i, k = k0 + tx;
        if (q < CRS && k < Kp) wt[static_cast<size_t>(q) * Kp + k] = tile[tx][i];
    }
}

__global__ __launch_bounds__(kWaves * 64)
void repack_filter_kernel(const float *__restrict__ w, int K, int Kp, int CRS, float *__restrict__ wt) {
    __shared__ float tile[64][65];
    repack_tile(w, K, Kp, CRS, wt, blockIdx.x, blockIdx.y, tile);
}

// Workgroups [0, groups) compact (grid-stride over planes) and store their
// count in parts[b]; workgroup 0 also zeroes parts[groups .. nparts).
// Workgroups from `groups` on repack one filter tile each.
__global__ __launch_bounds__(kWaves * 64)
void prep_kernel(const float *__restrict__ x, int planes, int H, int W, int32_t *__restrict__ row_ptr,
                 NzEntry *__restrict__ nz, uint32_t *__restrict__ parts, int groups, int nparts,
                 const float *__restrict__ w, int K, int Kp, int CRS, int qtiles, float *__restrict__ wt) {
    __shared__ float tile[64][65];
    __shared__ uint32_t wave_count[kWaves];
    const int b = blockIdx.x;
    if (b >= groups) {
        const int t = b - groups;
        repack_tile(w, K, Kp, CRS, wt, t % qtiles, t / qtiles, tile);
        return;
    }
    const int wave = threadIdx.x >> 6;
    const uint32_t listed = compact_planes(x, planes, H, W, row_ptr, nz, b * kWaves + wave, groups * kWaves);
    if ((threadIdx.x & 63) == 0) wave_count[wave] = listed;
    if (b == 0) {
        for (int i = groups + static_cast<int>(threadIdx.x); i < nparts; i += kWaves * 64) parts[i] = 0u;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t s = 0;
#pragma unroll
        for (int i = 0; i < kWaves; ++i) s += wave_count[i];
        parts[b] = s;
    }
}

// Nonzero count of x (total elements) in per-workgroup parts, for the
// sparse/dense decision when no compaction runs (ISC step 1's count without
// the list): workgroup b counts one contiguous chunk of whole 16-byte
// groups, eight of them in flight per thread (32 MB in flight over the
// launch: a cold read of AlexNet conv2's input in one round trip);
// workgroup 0 also counts
// the elements before the first 16-byte boundary and zeroes parts[groups ..
// nparts), the last one counts the elements after the last whole group.
// The workgroups past `groups` repack the filter, one 64 x 64 tile each.
constexpr int kCountWaves = 16;   // 1024 threads
constexpr int kCountUnroll = 8;   // 16-byte loads in flight per thread

__device__ __forceinline__ uint32_t nz4(const float4 &v) {
    return ((__float_as_uint(v.x) & 0x7fffffffu) != 0u) + ((__float_as_uint(v.y) & 0x7fffffffu) != 0u) +
           ((__float_as_uint(v.z) & 0x7fffffffu) != 0u) + ((__float_as_uint(v.w) & 0x7fffffffu) != 0u);
}

// Cache warm-up: workgroup `blk` reads its 64 KiB of p[0 .. n4) with four
// 16-byte loads in flight per thread.  The loaded words feed a value that
// is stored (to a word nobody reads) only when it equals `key`, so the loads
// are not dead code; what matters is that the lines end up cached.
constexpr int kWarmThreads = 1024, kWarmLoads = 4;
constexpr int64_t kWarmBytesPerGroup = static_cast<int64_t>(kWarmThreads) * kWarmLoads * 16;

__device__ __forceinline__ void warm_lines(const uint4 *__restrict__ p, int64_t n4, int64_t blk, uint32_t key,
                                           uint32_t *sink) {
    const int64_t base = blk * kWarmThreads * kWarmLoads + threadIdx.x;
    uint4 v[kWarmLoads];
#pragma unroll
    for (int j = 0; j < kWarmLoads; ++j) {
        const int64_t i = base + static_cast<int64_t>(j) * kWarmThreads;
        v[j] = p[i < n4 ? i : n4 - 1];
    }
    uint32_t acc = 0;
#pragma unroll
    for (int j = 0; j < kWarmLoads; ++j) acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
    if (acc == key) *sink = acc;
}

constexpr uint32_t kWarmKey = 0x5bd1e995u;

__global__ __launch_bounds__(kCountWaves * 64)
void count_parts_kernel(const float *__restrict__ x, int64_t total, int head, uint32_t *__restrict__ parts,
                        int groups, int nparts, const float *__restrict__ w, int K, int Kp, int CRS, int qtiles,
                        float *__restrict__ wt, const uint4 *__restrict__ warm, int64_t warm_n4, uint32_t *sink) {
    __shared__ uint32_t wave_count[kCountWaves];
    __shared__ float tile[64][65];
    const int b = blockIdx.x;
    if (b >= groups) {  // filter repack, one 64 x 64 tile per workgroup; or cache warm-up
        const int t = b - groups;
        if (w)
            repack_tile(w, K, Kp, CRS, wt, t % qtiles, t / qtiles, tile);
        else
            warm_lines(warm, warm_n4, t, kWarmKey, sink);
        return;
    }
    constexpr int kThreads = kCountWaves * 64;
    // x[head ..] is 16-byte aligned; n4 whole groups of four follow
    const int64_t n4 = (total - head) / 4;
    const float4 *x4 = reinterpret_cast<const float4 *>(x + head);
    const int64_t chunk = (n4 + groups - 1) / groups;
    const int64_t beg = b * chunk;
    const int64_t end = min(n4, beg + chunk);
    uint32_t cnt = 0;
    for (int64_t g0 = beg + threadIdx.x; g0 < end; g0 += static_cast<int64_t>(kThreads) * kCountUnroll) {
        float4 v[kCountUnroll];
#pragma unroll
        for (int u = 0; u < kCountUnroll; ++u) {
            const int64_t g = g0 + static_cast<int64_t>(u) * kThreads;
            v[u] = load_once(x4 + (g < end ? g : beg));  // past the end: an element already counted, not added
        }
#pragma unroll
        for (int u = 0; u < kCountUnroll; ++u)
            if (g0 + static_cast<int64_t>(u) * kThreads < end) cnt += nz4(v[u]);
    }
    if (b == 0 && static_cast<int>(threadIdx.x) < head)
        cnt += (__float_as_uint(x[threadIdx.x]) & 0x7fffffffu) != 0u;
    if (b == groups - 1) {
        const int64_t t0 = head + 4 * n4;  // at most 3 elements after the last whole group
        if (t0 + static_cast<int64_t>(threadIdx.x) < total)
            cnt += (__float_as_uint(x[t0 + threadIdx.x]) & 0x7fffffffu) != 0u;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off);
    if ((threadIdx.x & 63) == 0) wave_count[threadIdx.x >> 6] = cnt;
    if (b == 0) {
        for (int i = groups + static_cast<int>(threadIdx.x); i < nparts; i += kThreads) parts[i] = 0u;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t s = 0;
#pragma unroll
        for (int i = 0; i < kCountWaves; ++i) s += wave_count[i];
        parts[b] = s;
    }
}


// Workgroup 0 turns a census into the decision's parts: the census's counts
// summed with 16-byte loads (a census of a few thousand workgroups is read
// once, here, instead of by every wavefront of the next kernel); the other
// workgroups warm the cache with `warm`.
constexpr int kCensusThreads = kWarmThreads;

__global__ __launch_bounds__(kCensusThreads)
void census_parts_kernel(const CensusHeader *__restrict__ census, uint32_t cap, unsigned long long elems,
                         uint32_t *__restrict__ parts, const uint4 *__restrict__ warm, int64_t warm_n4,
                         uint32_t *sink) {
    if (blockIdx.x > 0) {
        warm_lines(warm, warm_n4, blockIdx.x - 1, kWarmKey, sink);
        return;
    }
    __shared__ unsigned long long part[kCensusThreads / 64];
    const CensusHeader h = *census;
    const bool ok = h.elems == elems && h.nslots <= cap && h.nslots % 4 == 0;
    unsigned long long s = 0;
    if (ok) {
        const uint4 *c4 = reinterpret_cast<const uint4 *>(census + 1);
        const int n4 = static_cast<int>(h.nslots / 4);
        for (int i0 = threadIdx.x; i0 < n4; i0 += 4 * kCensusThreads) {
            uint4 v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = c4[min(i0 + j * kCensusThreads, n4 - 1)];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (i0 + j * kCensusThreads < n4)
                    s += static_cast<unsigned long long>(v[j].x) + v[j].y + v[j].z + v[j].w;
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long t = 0;
#pragma unroll
        for (int i = 0; i < kCensusThreads / 64; ++i) t += part[i];
        // an unusable census, or (impossible for a real one) a total of 2^32
        // or more: all ones, which the decision reads as an unknown count
        const bool known = ok && t < (1ull << 32);
        parts[0] = known ? static_cast<uint32_t>(t) : 0xffffffffu;
        parts[1] = known ? 0u : 0xffffffffu;
        parts[2] = 0u;
        parts[3] = 0u;
    }
}

// The output epilogue as a pass of its own, for the kernels over compacted
// lists (which store y without one): y rectified in place and its nonzeros
// counted into the census; workgroup b takes one contiguous chunk.
__global__ __launch_bounds__(kWaves * 64)
void rectify_kernel(float *__restrict__ y, int64_t n, Epilogue epi, Decision dec) {
    if (!decision_gate(dec, 1u)) return;
    __shared__ uint32_t sums[kWaves];
    const int64_t chunk = (n + gridDim.x - 1) / gridDim.x;
    const int64_t beg = static_cast<int64_t>(blockIdx.x) * chunk;
    const int64_t end = min(n, beg + chunk);
    uint32_t cnt = 0;
    for (int64_t e = beg + threadIdx.x; e < end; e += kWaves * 64) {
        const float v = epilogue_value(y[e], epi.relu);
        cnt += nonzero_bit(v);
        y[e] = v;
    }
    if (epi.census) census_commit(epi, cnt, sums);
}

int compact_groups(int planes) {
    // one plane per wavefront while every wavefront can be resident at once
    // (24 per CU on 256 CUs), else as many planes per wavefront as it takes
    // (the loads of a wavefront's next plane fly while it lists the current
    // one)
    constexpr int kResidentWaves = 256 * 24;
    const int per_wave = std::max(1, (planes + kResidentWaves - 1) / kResidentWaves);
    const int waves = (planes + per_wave - 1) / per_wave;
    return std::max(1, (waves + kWaves - 1) / kWaves);
}

}  // namespace

hipError_t launch_compact(const float *x, int planes, int H, int W, int32_t *row_ptr,
                          NzEntry *nz, unsigned long long *counter, hipStream_t s) {
    compact_kernel<<<compact_groups(planes), kWaves * 64, 0, s>>>(x, planes, H, W, row_ptr, nz, counter);
    count_kernel<<<(planes + kCountThreads - 1) / kCountThreads, kCountThreads, 0, s>>>(row_ptr, planes, H, counter);
    return hipGetLastError();
}

hipError_t launch_census_parts(const CensusHeader *census, uint32_t cap, unsigned long long elems, uint32_t *parts,
                               const void *warm, size_t warm_bytes, Ctrl *ctrl, hipStream_t s) {
    // whole 16-byte words of the warmed range (a repacked filter is a
    // multiple of 64 floats)
    const int64_t n4 = warm ? static_cast<int64_t>(warm_bytes / 16) : 0;
    const int64_t groups = (n4 * 16 + kWarmBytesPerGroup - 1) / kWarmBytesPerGroup;
    census_parts_kernel<<<static_cast<unsigned>(1 + groups), kCensusThreads, 0, s>>>(
        census, cap, elems, parts, static_cast<const uint4 *>(warm), n4, &ctrl->sink);
    return hipGetLastError();
}

size_t repacked_filter_floats(int K, int C, int R, int S) {
    const size_t Kp = (static_cast<size_t>(K) + 63) / 64 * 64;
    return static_cast<size_t>(C) * R * S * Kp;
}

hipError_t launch_repack_filter(const float *w, int K, int C, int R, int S, float *wt, hipStream_t s) {
    const int CRS = C * R * S;
    const int Kp = (K + 63) / 64 * 64;
    dim3 grid((CRS + 63) / 64, Kp / 64);
    repack_filter_kernel<<<grid, kWaves * 64, 0, s>>>(w, K, Kp, CRS, wt);
    return hipGetLastError();
}

// At most 256 counting workgroups, so that the decision sums at most 256
// parts: one 16-byte load per lane of one wavefront.
constexpr int kCountGroups = 256;

hipError_t launch_count_parts(const float *x, int64_t total, uint32_t *parts, int *nparts, hipStream_t s,
                              const float *w, int K, int C, int R, int S, float *wt, const void *warm,
                              size_t warm_bytes, Ctrl *ctrl) {
    const int64_t per = static_cast<int64_t>(kCountWaves) * 64 * kCountUnroll * 4;  // elements per workgroup, at least
    const int groups = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(kCountGroups, (total + per - 1) / per)));
    const int np = (groups + 3) / 4 * 4;
    const int CRS = C * R * S;
    const int Kp = (K + 63) / 64 * 64;
    const int qtiles = (CRS + 63) / 64;
    const int64_t warm_n4 = !w && warm && ctrl ? static_cast<int64_t>(warm_bytes / 16) : 0;
    const int tiles = w ? qtiles * (Kp / 64)
                        : static_cast<int>((warm_n4 * 16 + kWarmBytesPerGroup - 1) / kWarmBytesPerGroup);
    // elements before the first 16-byte boundary (x is 4-byte aligned)
    const int head = static_cast<int>(std::min<int64_t>(
        total, ((16 - reinterpret_cast<uintptr_t>(x) % 16) % 16) / 4));
    count_parts_kernel<<<groups + tiles, kCountWaves * 64, 0, s>>>(
        x, total, head, parts, groups, np, w, K, Kp, CRS, qtiles, wt, static_cast<const uint4 *>(warm), warm_n4,
        ctrl ? &ctrl->sink : nullptr);
    *nparts = np;
    return hipGetLastError();
}

hipError_t launch_rectify(float *y, int64_t n, const Epilogue &epi, const Decision &dec, hipStream_t s) {
    const int64_t per = static_cast<int64_t>(kWaves) * 64 * 16;  // elements per workgroup, at least
    const int groups = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(kRectifyGroups, (n + per - 1) / per)));
    if (epi.census && census_slots_for(groups) > epi.cap) return hipErrorInvalidValue;
    rectify_kernel<<<groups, kWaves * 64, 0, s>>>(y, n, epi, dec);
    return hipGetLastError();
}

hipError_t launch_prep(const float *x, int planes, int H, int W, int32_t *row_ptr, NzEntry *nz,
                       uint32_t *parts, int *nparts, const float *w, int K, int C, int R, int S,
                       float *wt, hipStream_t s) {
    const int groups = std::min(compact_groups(planes), kMaxParts);
    const int np = (groups + 3) / 4 * 4;
    const int CRS = C * R * S;
    const int Kp = (K + 63) / 64 * 64;
    const int qtiles = (CRS + 63) / 64;
    const int tiles = qtiles * (Kp / 64);
    prep_kernel<<<groups + tiles, kWaves * 64, 0, s>>>(x, planes, H, W, row_ptr, nz, parts, groups, np, w, K, Kp,
                                                       CRS, qtiles, wt);
    *nparts = np;
    return hipGetLastError();
}

}  // namespace isc
