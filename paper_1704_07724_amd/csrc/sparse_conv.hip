// ISC steps 2 and 3 (Sec. "Sparse Convolution"), general kernel: zero-skipping
// convolution over the compacted nonzero lists with the output tile kept in
// LDS.  It handles every shape (any R x S, any stride); the register-tile
// kernel (sparse_reg.hip) is used instead where it applies.
//
// Layout of the work.  A workgroup owns one image n, one block of 64 output
// maps k, a band of output rows and a tile of output columns; each of its
// four wavefronts owns TH consecutive rows of the band.  Lanes run over k, as
// the paper's SIMD lanes do (step 2 multiplies one nonzero input by
// K-contiguous weights), so every nonzero input is a wave-uniform scalar and
// the only per-lane data are the weights and the accumulators.  A wavefront
// walks the nonzeros of the input rows that reach its output rows -- one
// contiguous slice of each plane's row-major list, found from the row
// offsets -- and for every nonzero and filter tap adds v * W[k, c, r, s] into
// an accumulator tile kept in LDS as [row][column][k], the "temporary
// results" of step 2.  The tile has halo columns, so taps that fall left or
// right of the output need no test at stride 1; rows outside the
// wavefront's band are skipped per filter row.  At the end the tile is read
// back transposed and stored to NCHW (step 3).
//
// Every accumulator element is updated only by its own lane, in list order,
// so results are deterministic run to run.
#include "isc_internal.hpp"

#include <algorithm>
#include <atomic>
#include <cstdlib>
#include <cstring>

namespace isc {
namespace {

constexpr int kLanes = 64;
constexpr int kAccStride = kLanes + 1;  // padded: transposed reads avoid bank conflicts
constexpr int kWaves = 4;               // wavefronts per workgroup

// wt: the repacked filter, wt[((c * R + r) * S + s) * Kp + k] (see
// launch_repack_filter).
struct SparseArgs {
    const int32_t *row_ptr;
    const NzEntry *nz;
    const float *wt;
    float *y;
    int N, C, H, W, K, Kp, R, S, T, P, Ho, Wo;
    int TH;       // output rows per wavefront
    int bands;    // row bands per image
    int TW;       // output columns per tile
    int ctiles;   // column tiles per image
    int kblocks;  // blocks of 64 output maps
    int WA;       // accumulator row width (tile columns plus halo)
    int hx;       // accumulator column of the tile's first output column
    Decision dec;
};

// Where a workgroup / wavefront sits in the output.
struct Tile {
    int n, kb, oy0, ox0, rows, cols;
    int ylo, yhi, xlo, xhi;  // input rows / columns whose taps reach the tile
    bool any;                // the wavefront owns at least one output
    bool whole_rows;         // the tile's input columns are the full rows
};

__device__ __forceinline__ Tile tile_of(const SparseArgs &a, int wave) {
    Tile t;
    int b = blockIdx.x;
    t.kb = b % a.kblocks;
    b /= a.kblocks;
    const int ct = b % a.ctiles;
    b /= a.ctiles;
    const int band = b % a.bands;
    t.n = b / a.bands;
    t.oy0 = (band * kWaves + wave) * a.TH;
    t.ox0 = ct * a.TW;
    t.rows = min(a.TH, a.Ho - t.oy0);
    t.cols = min(a.TW, a.Wo - t.ox0);
    t.ylo = max(0, t.oy0 * a.T - a.P);
    t.yhi = min(a.H - 1, (t.oy0 + t.rows - 1) * a.T - a.P + a.R - 1);
    t.xlo = max(0, t.ox0 * a.T - a.P);
    t.xhi = min(a.W - 1, (t.ox0 + t.cols - 1) * a.T - a.P + a.S - 1);
    t.any = t.rows > 0 && t.cols > 0 && t.ylo <= t.yhi;
    t.whole_rows = t.xlo == 0 && t.xhi == a.W - 1;
    return t;
}

// One nonzero input (value v at row yy, column xx of a channel's plane): add
// its products with that channel's filter taps w(r*S + s) (this lane's k)
// into the wavefront's accumulator tile.
template <int RT, int ST, typename WFn>
__device__ __forceinline__ void scatter_nonzero(const SparseArgs &a, const Tile &t, float *acc, int lane,
                                                WFn w, float v, int yy, int xx) {
    const int T = a.T, P = a.P, WA = a.WA, hx = a.hx;
    const int R = RT > 0 ? RT : a.R;
    const int S = ST > 0 ? ST : a.S;
    if (T == 1) {
        // accumulator column of tap s is col_last + (S - 1 - s): tap S-1 is
        // the leftmost, so every tap is a positive constant offset from one
        // address (the halo absorbs taps left or right of the tile)
        const int col_last = xx + P - t.ox0 + hx - (S - 1);
        if constexpr (RT > 0) {
#pragma unroll
            for (int r = 0; r < RT; ++r) {
                const int oy = yy + P - r - t.oy0;
                if (static_cast<unsigned>(oy) < static_cast<unsigned>(t.rows)) {
                    float *arow = acc + (oy * WA + col_last) * kAccStride + lane;
#pragma unroll
                    for (int s = 0; s < ST; ++s) {
                        float *p = arow + (ST - 1 - s) * kAccStride;
                        *p = __builtin_fmaf(v, w(r * ST + s), *p);
                    }
                }
            }
        } else {
            for (int r = 0; r < R; ++r) {
                const int oy = yy + P - r - t.oy0;
                if (static_cast<unsigned>(oy) >= static_cast<unsigned>(t.rows)) continue;
                float *arow = acc + (oy * WA + col_last) * kAccStride + lane;
                for (int s = 0; s < S; ++s) {
                    float *p = arow + (S - 1 - s) * kAccStride;
                    *p = __builtin_fmaf(v, w(r * S + s), *p);
                }
            }
        }
    } else {
        // general stride: a tap reaches output (oy, ox) only when its offset
        // divides by T (loops unrolled when R, S are compile-time, so the
        // weights stay in fixed registers)
#pragma unroll
        for (int r = 0; r < (RT > 0 ? RT : R); ++r) {
            const int ty = yy + P - r;
            if (ty < 0 || ty % T) continue;
            const int oy = ty / T - t.oy0;
            if (static_cast<unsigned>(oy) >= static_cast<unsigned>(t.rows)) continue;
#pragma unroll
            for (int s = 0; s < (ST > 0 ? ST : S); ++s) {
                const int tx = xx + P - s;
                if (tx < 0 || tx % T) continue;
                const int ox = tx / T - t.ox0;
                if (static_cast<unsigned>(ox) >= static_cast<unsigned>(t.cols)) continue;
                float *p = acc + (oy * WA + ox + hx) * kAccStride + lane;
                *p = __builtin_fmaf(v, w(r * S + s), *p);
            }
        }
    }
}

// Walk cnt entries of a wavefront-resident slice (lane j holds entry j).
template <int RT, int ST, typename WFn>
__device__ __forceinline__ void run_slice(const SparseArgs &a, const Tile &t, float *acc, int lane, WFn w,
                                          const NzEntry &mine, int cnt) {
    for (int j = 0; j < cnt; ++j) {
        const float v = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mine.v), j));
        const uint32_t yx = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(mine.yx), j));
        const int yy = static_cast<int>(yx >> 16);
        const int xx = static_cast<int>(yx & 0xffffu);
        if (!t.whole_rows && (xx < t.xlo || xx > t.xhi)) continue;
        scatter_nonzero<RT, ST>(a, t, acc, lane, w, v, yy, xx);
    }
}

__device__ __forceinline__ void zero_acc(float *acc, int positions, int lane) {
    for (int pos = 0; pos < positions; ++pos) acc[pos * kAccStride + lane] = 0.0f;
}

// Step 3: transpose the wavefront's [row][column][k] tile to NCHW; for a
// fixed k the rows x cols block is stored with consecutive lanes on
// consecutive columns (contiguous when the tile spans the output width).
__device__ __forceinline__ void write_tile(const SparseArgs &a, const Tile &t, const float *acc, int lane) {
    // other lanes' accumulators are read below: finish this wave's LDS writes
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (t.rows <= 0 || t.cols <= 0) return;
    const int count = t.rows * t.cols;
    const size_t plane_out = static_cast<size_t>(a.Ho) * a.Wo;
    const int kmax = min(kLanes, a.K - t.kb * kLanes);
    float *ybase = a.y + (static_cast<size_t>(t.n) * a.K + t.kb * kLanes) * plane_out;
    for (int i0 = 0; i0 < count; i0 += kLanes) {
        const int idx = i0 + lane;
        if (idx < count) {
            const int oy = idx / t.cols;
            const int ox = idx - oy * t.cols;
            const float *src = acc + (oy * a.WA + ox + a.hx) * kAccStride;
            float *dst = ybase + static_cast<size_t>(t.oy0 + oy) * a.Wo + t.ox0 + ox;
            for (int kk = 0; kk < kmax; ++kk) dst[static_cast<size_t>(kk) * plane_out] = src[kk];
        }
    }
}

__device__ __forceinline__ bool gate_and_record(const SparseArgs &a) { return decision_gate(a.dec, 1u); }

// ---------------------------------------------------------------------------
// Generic kernel: any R x S (runtime), one channel at a time, weights read
// per tap from the repacked filter.

__global__ __launch_bounds__(kWaves * kLanes)
void sparse_conv_generic_kernel(SparseArgs a) {
    if (!gate_and_record(a)) return;
    extern __shared__ float4 lds4[];
    const int lane = threadIdx.x & (kLanes - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kLanes);
    const Tile t = tile_of(a, wave);
    float *acc = reinterpret_cast<float *>(lds4) + static_cast<size_t>(wave) * a.TH * a.WA * kAccStride;
    zero_acc(acc, a.TH * a.WA, lane);
    if (t.any) {
        const int RS = a.R * a.S;
        const size_t HW = static_cast<size_t>(a.H) * a.W;
        const float *wk = a.wt + t.kb * kLanes + lane;  // this lane's k (zero padded to Kp)
        for (int c = 0; c < a.C; ++c) {
            const size_t plane = static_cast<size_t>(t.n) * a.C + c;
            const int32_t *rp = a.row_ptr + plane * (a.H + 1);
            const int eb = rp[t.ylo];
            const int ee = rp[t.yhi + 1];
            const float *wc = wk + static_cast<size_t>(c) * RS * a.Kp;
            auto wfn = [&](int tap) { return wc[static_cast<size_t>(tap) * a.Kp]; };
            const NzEntry *ent = a.nz + plane * HW;
            for (int e = eb; e < ee; e += kLanes)
                run_slice<0, 0>(a, t, acc, lane, wfn, ent[e + lane], min(kLanes, ee - e));
        }
    }
    write_tile(a, t, acc, lane);
}

// Raise a kernel's dynamic-LDS limit once (per process) to the largest size
// requested so far; later launches of that size or less call nothing.
template <typename Kern>
hipError_t ensure_lds(Kern kern, std::atomic<int> &granted, int bytes) {
    if (bytes <= 64 * 1024 || granted.load(std::memory_order_acquire) >= bytes) return hipSuccess;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e == hipSuccess) {
        int cur = granted.load(std::memory_order_relaxed);
        while (cur < bytes && !granted.compare_exchange_weak(cur, bytes)) {
        }
    }
    return e;
}

constexpr size_t kLdsBudget = 80 * 1024;   // per workgroup: two workgroups per CU
constexpr size_t kLdsMax = 160 * 1024;
constexpr int64_t kTargetWaves = 256 * 16;  // ~16 wavefronts per CU

size_t acc_bytes(int th, int wa) {
    return ((static_cast<size_t>(kWaves) * th * wa * kAccStride + 3) / 4) * sizeof(float4);
}

// Tiling for a shape, given the LDS the kernel needs besides the
// accumulators; false if no tile fits.
bool tiling_for(const SparseShape &sh, size_t extra, int *TH, int *bands, int *TW, int *ctiles, int *WA,
                int *hx) {
    if (extra >= kLdsBudget) return false;
    const size_t budget = kLdsBudget - extra;
    int tw = sh.Wo, wa = 0, h = 0;
    auto halo = [&](int w, int *wa_out, int *hx_out) {
        if (sh.T != 1) {
            *hx_out = 0;
            *wa_out = w;
        } else if (w == sh.Wo) {
            // taps reach output columns x + P - s in [P - S + 1, W - 1 + P]
            *hx_out = std::max(0, sh.S - 1 - sh.P);
            *wa_out = *hx_out + std::max(sh.Wo, sh.W + sh.P);
        } else {
            *hx_out = sh.S - 1;
            *wa_out = w + 2 * (sh.S - 1);
        }
    };
    halo(tw, &wa, &h);
    if (acc_bytes(1, wa) > budget) {
        const int fit = static_cast<int>(budget / (kWaves * kAccStride * sizeof(float))) - 1;
        tw = sh.T == 1 ? fit - 2 * (sh.S - 1) : fit;
        if (tw < 1) return false;
        halo(tw, &wa, &h);
    }
    // rows per wavefront: as many as LDS allows while the grid keeps about
    // 16 wavefronts per CU (other wavefronts hide each one's latencies)
    const int64_t kblocks = (sh.K + kLanes - 1) / kLanes;
    const int64_t ctl = (sh.Wo + tw - 1) / tw;
    int th = 1;
    for (int t = 2; t <= sh.Ho && acc_bytes(t, wa) <= budget; ++t) {
        const int64_t wavefronts = static_cast<int64_t>(sh.N) * ((sh.Ho + t - 1) / t) * ctl * kblocks;
        if (wavefronts < kTargetWaves) break;
        th = t;
    }
    const int bands0 = (sh.Ho + kWaves * th - 1) / (kWaves * th);
    th = (sh.Ho + bands0 * kWaves - 1) / (bands0 * kWaves);  // balance rows over wavefronts
    if (sh.tu.rows > 0) th = sh.tu.rows;
    if (acc_bytes(th, wa) + extra > kLdsMax) return false;
    *TH = th;
    *bands = (sh.Ho + kWaves * th - 1) / (kWaves * th);
    *TW = tw;
    *ctiles = (sh.Wo + tw - 1) / tw;
    *WA = wa;
    *hx = h;
    return true;
}

template <typename Kern>
hipError_t launch_with(Kern kern, std::atomic<int> &granted, const SparseArgs &a, size_t extra, hipStream_t s) {
    const size_t lds = acc_bytes(a.TH, a.WA) + extra;
    const int grid = a.N * a.bands * a.ctiles * a.kblocks;
    hipError_t e = ensure_lds(kern, granted, static_cast<int>(lds));
    if (e != hipSuccess) return e;
    kern<<<grid, kWaves * kLanes, lds, s>>>(a);
    return hipGetLastError();
}

}  // namespace

bool sparse_ring_applies(const SparseShape &sh);
hipError_t launch_sparse_ring(const SparseShape &sh, const int32_t *row_ptr, const NzEntry *nz, const float *wt,
                              float *y, const Decision &dec, hipStream_t s);
bool sparse_res_applies(const SparseShape &sh);
hipError_t launch_sparse_res(const SparseShape &sh, const int32_t *row_ptr, const NzEntry *nz, const float *wt,
                             float *y, const Decision &dec, hipStream_t s);

bool sparse_tiling(const SparseShape &sh, int *TH, int *bands, int *TW, int *ctiles, int *WA, int *hx) {
    return tiling_for(sh, 0, TH, bands, TW, ctiles, WA, hx);
}

bool sparse_conv_feasible(const SparseShape &sh) { return list_kernel_for(sh) != kListNone; }

int list_kernel_waves(int kernel) { return kernel == kListResident ? 16 : 4; }

// Kernel over compacted lists: the filter-resident register kernel when the
// filter of 64 output maps fits in LDS, else the filter-ring register kernel,
// else the LDS-accumulator kernel (any filter, any stride).
// A caller's tuning.kernel naming one of the three restricts the choice.
int list_kernel_for(const SparseShape &sh) {
    const int want = sh.tu.kernel;
    const bool any = want != kListResident && want != kListRing && want != kListGeneric;
    if ((any || want == kListResident) && sparse_res_applies(sh)) return kListResident;
    if ((any || want == kListRing) && sparse_ring_applies(sh)) return kListRing;
    int th, bands, tw, ct, wa, hx;
    return tiling_for(sh, 0, &th, &bands, &tw, &ct, &wa, &hx) ? kListGeneric : kListNone;
}

hipError_t launch_sparse_conv(const SparseShape &sh, const int32_t *row_ptr, const NzEntry *nz,
                              const float *wt, float *y, const Decision &dec, hipStream_t s) {
    const int which = list_kernel_for(sh);
    if (which == kListResident) return launch_sparse_res(sh, row_ptr, nz, wt, y, dec, s);
    if (which == kListRing) return launch_sparse_ring(sh, row_ptr, nz, wt, y, dec, s);
    if (which == kListNone) return hipErrorInvalidValue;
    SparseArgs a{};
    a.row_ptr = row_ptr;
    a.nz = nz;
    a.wt = wt;
    a.y = y;
    a.N = sh.N; a.C = sh.C; a.H = sh.H; a.W = sh.W; a.K = sh.K; a.Kp = (sh.K + kLanes - 1) / kLanes * kLanes;
    a.R = sh.R; a.S = sh.S; a.T = sh.T; a.P = sh.P; a.Ho = sh.Ho; a.Wo = sh.Wo;
    a.dec = dec;
    if (!tiling_for(sh, 0, &a.TH, &a.bands, &a.TW, &a.ctiles, &a.WA, &a.hx)) return hipErrorInvalidValue;
    a.kblocks = (sh.K + kLanes - 1) / kLanes;
    static std::atomic<int> granted{0};
    return launch_with(sparse_conv_generic_kernel, granted, a, 0, s);
}

}  // namespace isc
