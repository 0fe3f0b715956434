// ISC steps 2 and 3 (Sec. "Sparse Convolution"): zero-skipping convolution
// over the compacted nonzero lists, output-stationary per workgroup.
//
// Layout of the work.  A workgroup owns one image n, one block of 64 output
// maps k, a band of output rows and a tile of output columns; each of its
// wavefronts owns TH consecutive rows of the band.  Lanes run over k, as the
// paper's SIMD lanes do (step 2 multiplies one nonzero input by K-contiguous
// weights), so every nonzero input is a wave-uniform scalar and the only
// per-lane data are the weights and the accumulators.  The wavefront walks
// the nonzeros of the input rows that reach its output rows -- one
// contiguous slice of the plane's row-major list, found from the row
// offsets -- and for every nonzero and every filter tap adds v * W[k,c,r,s]
// into an accumulator tile kept in LDS as [row][column][k], the "temporary
// results" of step 2.  The tile has halo columns, so taps that fall left or
// right of the output need no test at stride 1; rows outside the wavefront's
// band are skipped per filter row.  At the end the tile is read back
// transposed and stored to NCHW (step 3).
//
// Filter weights come from the repacked [C][R][S][K] copy (the paper's
// column-major kernel matrix): for a channel c the R*S weights of the lane's
// k sit in registers, loaded one channel ahead.
//
// Every accumulator element is updated only by its own lane, in the order of
// the nonzero list, so results are deterministic run to run.
#include "isc_internal.hpp"

#include <algorithm>
#include <atomic>
#include <cstdlib>

namespace isc {
namespace {

constexpr int kLanes = 64;
constexpr int kAccStride = kLanes + 1;  // padded: transposed reads avoid bank conflicts

struct SparseArgs {
    const int32_t *row_ptr;
    const NzEntry *nz;
    const float *wt;  // [C][R][S][K]
    float *y;
    int N, C, H, W, K, R, S, T, P, Ho, Wo;
    int TH;       // output rows per wavefront
    int bands;    // row bands per image
    int TW;       // output columns per tile
    int ctiles;   // column tiles per image
    int kblocks;  // blocks of 64 output maps
    int WA;       // accumulator row width (tile columns plus halo)
    int hx;       // accumulator column of the tile's first output column
    Decision dec;
};

// acc += v * w on the lane's own accumulator; kAtomic selects an LDS atomic
// add (no read-back, fire and forget) instead of load / fma / store.
template <bool kAtomic>
__device__ __forceinline__ void acc_add(float *p, float v, float w) {
    if constexpr (kAtomic) {
        __hip_atomic_fetch_add(p, v * w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
    } else {
        *p = __builtin_fmaf(v, w, *p);
    }
}

template <int RT, int ST, bool kAtomic>
__global__ __launch_bounds__(256)
void sparse_conv_kernel(SparseArgs a) {
    const bool run = decision_says_run(a.dec);
    if (blockIdx.x == 0 && threadIdx.x == 0 && a.dec.record) a.dec.record->path_taken = run ? 1u : 2u;
    if (!run) return;

    extern __shared__ float lds[];
    const int lane = threadIdx.x & (kLanes - 1);
    const int wave = threadIdx.x / kLanes;
    const int waves = blockDim.x / kLanes;

    constexpr int kRegRS = RT * ST;  // weights held in registers (0: read per tap)
    const int R = RT > 0 ? RT : a.R;
    const int S = ST > 0 ? ST : a.S;
    const int RS = R * S;
    const int T = a.T, P = a.P, H = a.H, W = a.W, K = a.K;
    const int Ho = a.Ho, Wo = a.Wo, TH = a.TH, WA = a.WA, hx = a.hx;

    int b = blockIdx.x;
    const int kb = b % a.kblocks;
    b /= a.kblocks;
    const int ct = b % a.ctiles;
    b /= a.ctiles;
    const int band = b % a.bands;
    const int n = b / a.bands;

    const int oy0 = (band * waves + wave) * TH;  // first output row of this wavefront
    const int ox0 = ct * a.TW;                   // first output column of the tile
    const int k = kb * kLanes + lane;
    const bool k_ok = k < K;

    float *acc = lds + static_cast<size_t>(wave) * TH * WA * kAccStride;
    for (int pos = 0; pos < TH * WA; ++pos) acc[pos * kAccStride + lane] = 0.0f;

    const int rows = min(TH, Ho - oy0);      // rows this wavefront owns
    const int cols = min(a.TW, Wo - ox0);    // columns of this tile
    if (rows > 0) {
        // input rows / columns whose taps reach the owned outputs
        const int ylo = max(0, oy0 * T - P);
        const int yhi = min(H - 1, (oy0 + rows - 1) * T - P + R - 1);
        const int xlo = max(0, ox0 * T - P);
        const int xhi = min(W - 1, (ox0 + cols - 1) * T - P + S - 1);
        const bool whole_rows = xlo == 0 && xhi == W - 1;
        const size_t HW = static_cast<size_t>(H) * W;

        float wcur[kRegRS > 0 ? kRegRS : 1];
        float wnext[kRegRS > 0 ? kRegRS : 1];
        if constexpr (kRegRS > 0) {
#pragma unroll
            for (int t = 0; t < kRegRS; ++t)
                wcur[t] = k_ok ? a.wt[static_cast<size_t>(t) * K + k] : 0.0f;
        }

        for (int c = 0; c < a.C; ++c) {
            if constexpr (kRegRS > 0) {
                if (c + 1 < a.C) {
                    const float *wn = a.wt + static_cast<size_t>(c + 1) * kRegRS * K;
#pragma unroll
                    for (int t = 0; t < kRegRS; ++t)
                        wnext[t] = k_ok ? wn[static_cast<size_t>(t) * K + k] : 0.0f;
                }
            }
            const size_t plane = static_cast<size_t>(n) * a.C + c;
            const int32_t *rp = a.row_ptr + plane * (H + 1);
            const int e_begin = ylo <= yhi ? rp[ylo] : 0;
            const int e_end = ylo <= yhi ? rp[yhi + 1] : 0;
            const NzEntry *ent = a.nz + plane * HW;
            const float *wc = a.wt + static_cast<size_t>(c) * RS * K;

            for (int e = e_begin; e < e_end; ++e) {
                const NzEntry q = ent[e];
                const float v = q.v;
                const int yy = static_cast<int>(q.yx >> 16);
                const int xx = static_cast<int>(q.yx & 0xffffu);
                if (!whole_rows && (xx < xlo || xx > xhi)) continue;
                if (T == 1) {
                    // accumulator column of tap s is col_s0 - s (halo absorbs
                    // taps left or right of the tile)
                    const int col_s0 = xx + P - ox0 + hx;
                    if constexpr (kRegRS > 0) {
#pragma unroll
                        for (int r = 0; r < RT; ++r) {
                            const int oy = yy + P - r - oy0;
                            if (static_cast<unsigned>(oy) < static_cast<unsigned>(rows)) {
                                float *arow = acc + (oy * WA + col_s0) * kAccStride + lane;
#pragma unroll
                                for (int s = 0; s < ST; ++s)
                                    acc_add<kAtomic>(arow - s * kAccStride, v, wcur[r * ST + s]);
                            }
                        }
                    } else {
                        for (int r = 0; r < R; ++r) {
                            const int oy = yy + P - r - oy0;
                            if (static_cast<unsigned>(oy) >= static_cast<unsigned>(rows)) continue;
                            float *arow = acc + (oy * WA + col_s0) * kAccStride + lane;
                            for (int s = 0; s < S; ++s) {
                                const float wv = k_ok ? wc[static_cast<size_t>(r * S + s) * K + k] : 0.0f;
                                acc_add<kAtomic>(arow - s * kAccStride, v, wv);
                            }
                        }
                    }
                } else {
                    // general stride: a tap reaches output (oy, ox) only when
                    // its offset divides by T
                    for (int r = 0; r < R; ++r) {
                        const int ty = yy + P - r;
                        if (ty < 0 || ty % T) continue;
                        const int oy = ty / T - oy0;
                        if (static_cast<unsigned>(oy) >= static_cast<unsigned>(rows)) continue;
                        for (int s = 0; s < S; ++s) {
                            const int tx = xx + P - s;
                            if (tx < 0 || tx % T) continue;
                            const int ox = tx / T - ox0;
                            if (static_cast<unsigned>(ox) >= static_cast<unsigned>(cols)) continue;
                            float wv;
                            if constexpr (kRegRS > 0) {
                                wv = wcur[r * ST + s];
                            } else {
                                wv = k_ok ? wc[static_cast<size_t>(r * S + s) * K + k] : 0.0f;
                            }
                            acc_add<kAtomic>(acc + (oy * WA + ox + hx) * kAccStride + lane, v, wv);
                        }
                    }
                }
            }
            if constexpr (kRegRS > 0) {
#pragma unroll
                for (int t = 0; t < kRegRS; ++t) wcur[t] = wnext[t];
            }
        }
    }

    // other lanes' accumulators are read below: finish this wave's LDS writes
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    if (rows > 0 && cols > 0) {
        // step 3: transpose [row][column][k] -> NCHW; for a fixed k the
        // wavefront stores its rows x cols block, contiguous when the tile
        // spans the full output width
        const int count = rows * cols;
        const size_t plane_out = static_cast<size_t>(Ho) * Wo;
        const int kmax = min(kLanes, K - kb * kLanes);
        float *ybase = a.y + (static_cast<size_t>(n) * K + kb * kLanes) * plane_out;
        for (int i0 = 0; i0 < count; i0 += kLanes) {
            const int idx = i0 + lane;
            if (idx < count) {
                const int oy = idx / cols;
                const int ox = idx - oy * cols;
                const float *src = acc + (oy * WA + ox + hx) * kAccStride;
                float *dst = ybase + static_cast<size_t>(oy0 + oy) * Wo + ox0 + ox;
                for (int kk = 0; kk < kmax; ++kk) dst[static_cast<size_t>(kk) * plane_out] = src[kk];
            }
        }
    }
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

template <int RT, int ST>
hipError_t launch_sparse_t(const SparseArgs &a, int waves, bool atomic, hipStream_t s) {
    static std::atomic<int> granted_plain{0}, granted_atomic{0};
    const size_t lds = static_cast<size_t>(waves) * a.TH * a.WA * kAccStride * sizeof(float);
    const int grid = a.N * a.bands * a.ctiles * a.kblocks;
    auto kern = atomic ? sparse_conv_kernel<RT, ST, true> : sparse_conv_kernel<RT, ST, false>;
    hipError_t e = ensure_lds(kern, atomic ? granted_atomic : granted_plain, static_cast<int>(lds));
    if (e != hipSuccess) return e;
    kern<<<grid, waves * kLanes, lds, s>>>(a);
    return hipGetLastError();
}

constexpr size_t kLdsBudget = 80 * 1024;  // per workgroup: two workgroups per CU
constexpr int kWaves = 4;

}  // namespace

// Tiling of the sparse kernel for a shape; false if no tile fits in LDS.
bool sparse_tiling(const SparseShape &sh, int *TH, int *bands, int *TW, int *ctiles, int *WA, int *hx) {
    const size_t per_col = static_cast<size_t>(kAccStride) * sizeof(float);
    int tw = sh.Wo, wa, h;
    auto halo = [&](int t, int *wa_out, int *hx_out) {
        if (sh.T != 1) {
            *hx_out = 0;
            *wa_out = t;
        } else if (t == sh.Wo) {
            // taps reach output columns x + P - s in [P - S + 1, W - 1 + P]
            *hx_out = std::max(0, sh.S - 1 - sh.P);
            *wa_out = *hx_out + std::max(sh.Wo, sh.W + sh.P);
        } else {
            *hx_out = sh.S - 1;
            *wa_out = t + 2 * (sh.S - 1);
        }
    };
    halo(tw, &wa, &h);
    if (kWaves * wa * per_col > kLdsBudget) {
        const int fit = static_cast<int>(kLdsBudget / (kWaves * per_col));
        tw = sh.T == 1 ? fit - 2 * (sh.S - 1) : fit;
        if (tw < 1) return false;
        halo(tw, &wa, &h);
    }
    const size_t per_row = static_cast<size_t>(wa) * per_col;
    int th = static_cast<int>(kLdsBudget / (kWaves * per_row));
    th = std::max(1, std::min(th, (sh.Ho + kWaves - 1) / kWaves));
    const int bands0 = (sh.Ho + kWaves * th - 1) / (kWaves * th);
    th = (sh.Ho + bands0 * kWaves - 1) / (bands0 * kWaves);  // balance rows over wavefronts
    if (const char *env = std::getenv("ISC_SPARSE_TH")) th = std::max(1, std::atoi(env));
    if (kWaves * th * per_row > 160 * 1024) return false;
    *TH = th;
    *bands = (sh.Ho + kWaves * th - 1) / (kWaves * th);
    *TW = tw;
    *ctiles = (sh.Wo + tw - 1) / tw;
    *WA = wa;
    *hx = h;
    return true;
}

hipError_t launch_sparse_conv(const SparseShape &sh, const int32_t *row_ptr, const NzEntry *nz,
                              const float *wt, float *y, const Decision &dec, hipStream_t s) {
    SparseArgs a{};
    a.row_ptr = row_ptr;
    a.nz = nz;
    a.wt = wt;
    a.y = y;
    a.N = sh.N; a.C = sh.C; a.H = sh.H; a.W = sh.W; a.K = sh.K;
    a.R = sh.R; a.S = sh.S; a.T = sh.T; a.P = sh.P; a.Ho = sh.Ho; a.Wo = sh.Wo;
    a.dec = dec;
    if (!sparse_tiling(sh, &a.TH, &a.bands, &a.TW, &a.ctiles, &a.WA, &a.hx)) return hipErrorInvalidValue;
    a.kblocks = (sh.K + kLanes - 1) / kLanes;
    const char *env = std::getenv("ISC_SPARSE_ATOMIC");
    const bool atomic = env ? std::atoi(env) != 0 : false;

    if (sh.R == 1 && sh.S == 1) return launch_sparse_t<1, 1>(a, kWaves, atomic, s);
    if (sh.R == 3 && sh.S == 3) return launch_sparse_t<3, 3>(a, kWaves, atomic, s);
    if (sh.R == 5 && sh.S == 5) return launch_sparse_t<5, 5>(a, kWaves, atomic, s);
    if (sh.R == 7 && sh.S == 7) return launch_sparse_t<7, 7>(a, kWaves, atomic, s);
    return launch_sparse_t<0, 0>(a, kWaves, atomic, s);
}

// --- filter repack ----------------------------------------------------------

namespace {
__global__ __launch_bounds__(256)
void repack_filter_kernel(const float *__restrict__ w, int K, int CRS, float *__restrict__ wt) {
    // wt[q][k] = w[k][q] through a 64 x 64 LDS tile, both sides coalesced
    __shared__ float tile[64][65];
    const int q0 = blockIdx.x * 64, k0 = blockIdx.y * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4) {
        const int kk = k0 + i, q = q0 + tx;
        tile[i][tx] = (kk < K && q < CRS) ? w[static_cast<size_t>(kk) * CRS + q] : 0.0f;
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
        const int q = q0 + i, kk = k0 + tx;
        if (q < CRS && kk < K) wt[static_cast<size_t>(q) * K + kk] = tile[tx][i];
    }
}
}  // namespace

hipError_t launch_repack_filter(const float *w, int K, int CRS, float *wt, hipStream_t s) {
    dim3 grid((CRS + 63) / 64, (K + 63) / 64);
    repack_filter_kernel<<<grid, 256, 0, s>>>(w, K, CRS, wt);
    return hipGetLastError();
}

}  // namespace isc
