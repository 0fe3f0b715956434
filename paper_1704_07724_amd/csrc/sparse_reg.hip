// ISC steps 2 and 3 (Sec. "Sparse Convolution") with the output tile in
// registers: the fast kernel for stride 1 and square 1x1, 3x3, 5x5 filters.
//
// A wavefront owns one output row, a tile of up to TWM output columns and
// 64 * KPL output maps: lane l accumulates maps kbase + l*KPL + j (j < KPL)
// in registers acc[column][j].  Lanes run over k, as the paper's SIMD lanes
// do (step 2 multiplies one nonzero by K-contiguous weights), so each nonzero
// input is a wave-uniform scalar.  For filter row r the wavefront reads the
// row's weights w[s][j] from LDS into registers and walks the nonzeros of the
// matching input row (a contiguous run of the plane's row-major list).  A
// nonzero at column x adds v * w[s][j] to output column x + P - s for every
// tap s: the column is dynamic, but a compile-time binary dispatch on
// x + P selects a straight-line block whose register indices are constants,
// so the inner loop has no memory operations at all -- S * KPL fused
// multiply-adds per nonzero plus a few scalar compares.
//
// The workgroup's four wavefronts own four consecutive output rows of one
// image and share the filter: channel by channel the workgroup copies the
// channel's R*S*64*KPL weights into LDS, and each wavefront its nonzero run
// for that channel (both loaded into registers while the previous channel is
// computed), so the compute phase reads only LDS and registers.  At the end each lane stores its
// accumulators to NCHW (step 3).  Summation order per output is fixed (list
// order within a channel, channels in order), so results are deterministic.
#include "isc_internal.hpp"

#include <algorithm>
#include <cstdlib>

namespace isc {
namespace {

constexpr int kLanes = 64;
constexpr int kWaves = 4;
constexpr int kRunMax = 256;  // longest nonzero run (R input rows) a wavefront stages

struct RegArgs {
    const int32_t *row_ptr;
    const NzEntry *nz;
    const float *wt;  // [C][R][S][Kp], K contiguous
    float *y;
    int N, C, H, W, K, Kp, P, Ho, Wo;
    int TW;       // output columns per tile (<= TWM)
    int ctiles;   // column tiles per row
    int bands;    // groups of kWaves output rows
    int kgroups;  // groups of 64 * KPL output maps
    Decision dec;
};

// Nonzero at (shifted) column XP: taps s reach output column XP - s.
template <int S, int KPL, int TWM, int XP>
__device__ __forceinline__ void tap_block(float (&acc)[TWM][KPL], const float (&w)[S][KPL], float v) {
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const int ox = XP - s;
        if (ox >= 0 && ox < TWM) {
#pragma unroll
            for (int j = 0; j < KPL; ++j) acc[ox][j] = __builtin_fmaf(v, w[s][j], acc[ox][j]);
        }
    }
}

// Binary dispatch of xp in [LO, HI) onto the straight-line blocks.
template <int S, int KPL, int TWM, int LO, int HI>
__device__ __forceinline__ void dispatch(int xp, float (&acc)[TWM][KPL], const float (&w)[S][KPL], float v) {
    if constexpr (HI - LO == 1) {
        tap_block<S, KPL, TWM, LO>(acc, w, v);
    } else {
        constexpr int MID = (LO + HI) / 2;
        if (xp < MID)
            dispatch<S, KPL, TWM, LO, MID>(xp, acc, w, v);
        else
            dispatch<S, KPL, TWM, MID, HI>(xp, acc, w, v);
    }
}

template <int RS_, int KPL, int TWM>
__global__ __launch_bounds__(kWaves * kLanes)
void sparse_conv_reg_kernel(RegArgs a) {
    constexpr int R = RS_, S = RS_;
    constexpr int XMAX = TWM + S - 1;             // shifted columns a tile can see
    constexpr int KW = kLanes * KPL;              // output maps per wavefront
    constexpr int WF4 = R * S * KW / 4;           // float4 of one channel's weights
    constexpr int WPT = (WF4 + kWaves * kLanes - 1) / (kWaves * kLanes);
    constexpr int NOFF = R + 1;                   // row offsets kept per channel
    constexpr int EPL = kRunMax / kLanes;         // staged run entries per lane

    const bool run = decision_says_run(a.dec);
    if (blockIdx.x == 0 && threadIdx.x == 0 && a.dec.record) a.dec.record->path_taken = run ? 1u : 2u;
    if (!run) return;

    // LDS: one channel's weights [R*S][KW] | each wavefront's staged nonzero
    // run [kRunMax] | each wavefront's row offsets [C][R+1]
    extern __shared__ float4 lds4[];
    float *wlds = reinterpret_cast<float *>(lds4);
    const int lane = threadIdx.x & (kLanes - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kLanes);
    NzEntry *ebuf = reinterpret_cast<NzEntry *>(lds4 + WF4) + wave * kRunMax;
    int32_t *offs = reinterpret_cast<int32_t *>(reinterpret_cast<NzEntry *>(lds4 + WF4) + kWaves * kRunMax) +
                    wave * a.C * NOFF;

    int b = blockIdx.x;
    const int kg = b % a.kgroups;
    b /= a.kgroups;
    const int ct = b % a.ctiles;
    b /= a.ctiles;
    const int band = b % a.bands;
    const int n = b / a.bands;
    const int oy = band * kWaves + wave;
    const int ox0 = ct * a.TW;
    const int kbase = kg * KW;
    const int C = a.C, H = a.H, P = a.P;
    const bool row_ok = oy < a.Ho;
    // input rows oy + r - P for r in [0, R), clipped to the map
    const int ylo = max(0, oy - P);
    const int yhi = min(H - 1, oy - P + R - 1);
    const int nrows = row_ok ? max(0, yhi - ylo + 1) : 0;
    const int tw = min(a.TW, a.Wo - ox0);
    const int xlo = max(0, ox0 - P);
    const int xhi = min(a.W - 1, ox0 + tw - 1 - P + S - 1);
    const bool whole_rows = xlo == 0 && xhi == a.W - 1;
    const size_t HW = static_cast<size_t>(H) * a.W;
    const NzEntry *nz_n = a.nz + static_cast<size_t>(n) * C * HW;

    // row offsets of this wavefront's input rows, every channel, into LDS
    {
        const int32_t *rp_n = a.row_ptr + static_cast<size_t>(n) * C * (H + 1);
        for (int idx = lane; idx < C * NOFF; idx += kLanes) {
            const int c = idx / NOFF;
            const int i = idx - c * NOFF;
            offs[idx] = i <= nrows && nrows > 0 ? rp_n[static_cast<size_t>(c) * (H + 1) + ylo + i] : 0;
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }

    float acc[TWM][KPL];
#pragma unroll
    for (int x = 0; x < TWM; ++x)
#pragma unroll
        for (int j = 0; j < KPL; ++j) acc[x][j] = 0.0f;

    // one channel's weights, [R*S][KW] with k = kbase + lane*KPL + j, as
    // float4 runs of the K-contiguous filter (zero past Kp)
    float4 wst[WPT];
    auto load_weights = [&](int c) {
#pragma unroll
        for (int q = 0; q < WPT; ++q) {
            const int f = threadIdx.x + q * kWaves * kLanes;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (f < WF4) {
                const int tap = f / (KW / 4);
                const int k4 = kbase + 4 * (f - tap * (KW / 4));
                if (k4 < a.Kp)
                    v = *reinterpret_cast<const float4 *>(a.wt + (static_cast<size_t>(c) * R * S + tap) * a.Kp + k4);
            }
            wst[q] = v;
        }
    };
    auto store_weights = [&]() {
#pragma unroll
        for (int q = 0; q < WPT; ++q) {
            const int f = threadIdx.x + q * kWaves * kLanes;
            if (f < WF4) lds4[f] = wst[q];
        }
    };
    // this wavefront's nonzero run of channel c (at most kRunMax entries:
    // the kernel is used only when R * W <= kRunMax), lane-strided
    NzEntry est[EPL];
    auto load_run = [&](int c) {
        const int e0 = __builtin_amdgcn_readfirstlane(offs[c * NOFF]);
        const int cnt = __builtin_amdgcn_readfirstlane(offs[c * NOFF + nrows]) - e0;
        const NzEntry *src = nz_n + static_cast<size_t>(c) * HW + e0;
#pragma unroll
        for (int q = 0; q < EPL; ++q) {
            NzEntry m{0.0f, 0u};
            if (q * kLanes + lane < cnt) m = src[q * kLanes + lane];
            est[q] = m;
        }
    };
    auto store_run = [&]() {
#pragma unroll
        for (int q = 0; q < EPL; ++q) ebuf[q * kLanes + lane] = est[q];
    };

    load_weights(0);
    load_run(0);
    store_weights();
    store_run();
    __syncthreads();

    for (int c = 0; c < C; ++c) {
        // prefetch channel c + 1 into registers; the compute below reads
        // only LDS and registers that no load in flight writes
        if (c + 1 < C) {
            load_weights(c + 1);
            load_run(c + 1);
        }
        const int *oc = offs + c * NOFF;
        const int e0 = __builtin_amdgcn_readfirstlane(oc[0]);
        const int e_all = __builtin_amdgcn_readfirstlane(oc[nrows]) - e0;
        if (e_all > 0) {
            // one copy of the dispatch code: filter rows run as a loop, the
            // row's weights reloaded into the same registers
#pragma unroll 1
            for (int r = 0; r < R; ++r) {
                const int y = oy + r - P;
                if (y < ylo || y > yhi) continue;
                const int lo = __builtin_amdgcn_readfirstlane(oc[y - ylo]) - e0;
                const int hi = __builtin_amdgcn_readfirstlane(oc[y - ylo + 1]) - e0;
                if (hi <= lo) continue;
                float w[S][KPL];
#pragma unroll
                for (int s = 0; s < S; ++s)
#pragma unroll
                    for (int j = 0; j < KPL; ++j) w[s][j] = wlds[(r * S + s) * KW + lane * KPL + j];
#pragma unroll 1
                for (int q0 = lo & ~(kLanes - 1); q0 < hi; q0 += kLanes) {
                    const NzEntry mine = ebuf[q0 + lane];
                    const int jlo = max(lo, q0) - q0, jhi = min(hi, q0 + kLanes) - q0;
#pragma unroll 1
                    for (int jj = jlo; jj < jhi; ++jj) {
                        const float v = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mine.v), jj));
                        const int x = __builtin_amdgcn_readlane(static_cast<int>(mine.yx), jj) & 0xffff;
                        if (static_cast<unsigned>(x - xlo) > static_cast<unsigned>(xhi - xlo)) continue;
                        dispatch<S, KPL, TWM, 0, XMAX>(x + P - ox0, acc, w, v);
                    }
                }
            }
        }
        __syncthreads();
        if (c + 1 < C) {
            store_weights();
            store_run();
        }
        __syncthreads();
    }

    // step 3: each lane stores its accumulators to NCHW
    if (row_ok) {
        const size_t plane_out = static_cast<size_t>(a.Ho) * a.Wo;
        float *yrow = a.y + static_cast<size_t>(n) * a.K * plane_out + static_cast<size_t>(oy) * a.Wo + ox0;
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            const int k = kbase + lane * KPL + j;
            if (k < a.K) {
                float *dst = yrow + static_cast<size_t>(k) * plane_out;
#pragma unroll
                for (int x = 0; x < TWM; ++x)
                    if (x < tw) dst[x] = acc[x][j];
            }
        }
    }
}

// Output maps per lane for K (and filter width S).
int kpl_for(int K, int S) {
    if (K <= 64) return 1;
    if (K <= 128) return 2;
    if (K <= 256 || S >= 5) return 4;
    return 6;
}

int twm_for(int Wo) { return Wo <= 8 ? 8 : (Wo <= 16 ? 16 : 28); }

template <int RS_, int KPL, int TWM>
hipError_t launch_reg_t(const RegArgs &a, hipStream_t s) {
    constexpr size_t wbytes = sizeof(float) * RS_ * RS_ * kLanes * KPL;
    const size_t lds = wbytes + sizeof(NzEntry) * kWaves * kRunMax + sizeof(int32_t) * kWaves * a.C * (RS_ + 1);
    if (lds > 160 * 1024) return hipErrorInvalidValue;
    auto kern = sparse_conv_reg_kernel<RS_, KPL, TWM>;
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (e != hipSuccess) return e;
    }
    const int grid = a.N * a.bands * a.ctiles * a.kgroups;
    kern<<<grid, kWaves * kLanes, lds, s>>>(a);
    return hipGetLastError();
}

template <int RS_, int TWM>
hipError_t launch_reg_kpl(const RegArgs &a, int kpl, hipStream_t s) {
    switch (kpl) {
    case 1: return launch_reg_t<RS_, 1, TWM>(a, s);
    case 2: return launch_reg_t<RS_, 2, TWM>(a, s);
    case 4: return launch_reg_t<RS_, 4, TWM>(a, s);
    default:
        if constexpr (RS_ <= 3) return launch_reg_t<RS_, 6, TWM>(a, s);
        return hipErrorInvalidValue;
    }
}

template <int RS_>
hipError_t launch_reg_rs(const RegArgs &a, int kpl, int twm, hipStream_t s) {
    switch (twm) {
    case 8: return launch_reg_kpl<RS_, 8>(a, kpl, s);
    case 16: return launch_reg_kpl<RS_, 16>(a, kpl, s);
    default: return launch_reg_kpl<RS_, 28>(a, kpl, s);
    }
}

}  // namespace

bool sparse_reg_applies(const SparseShape &sh) {
    if (sh.T != 1 || sh.R != sh.S || !(sh.R == 1 || sh.R == 3 || sh.R == 5)) return false;
    // a wavefront's run (R whole input rows) must fit the staging buffer
    if (static_cast<int64_t>(sh.R) * sh.W > kRunMax) return false;
    // LDS: one channel's weights, the staged runs, the row offsets
    const size_t kw = static_cast<size_t>(kLanes) * kpl_for(sh.K, sh.S);
    const size_t lds = sizeof(float) * sh.R * sh.S * kw + sizeof(NzEntry) * kWaves * kRunMax +
                       sizeof(int32_t) * kWaves * sh.C * (sh.R + 1);
    return lds <= 160 * 1024;
}

hipError_t launch_sparse_reg(const SparseShape &sh, const int32_t *row_ptr, const NzEntry *nz, const float *wt,
                             float *y, const Decision &dec, hipStream_t s) {
    RegArgs a{};
    a.row_ptr = row_ptr;
    a.nz = nz;
    a.wt = wt;
    a.y = y;
    a.N = sh.N; a.C = sh.C; a.H = sh.H; a.W = sh.W; a.K = sh.K;
    a.Kp = (sh.K + kLanes - 1) / kLanes * kLanes;
    a.P = sh.P; a.Ho = sh.Ho; a.Wo = sh.Wo;
    const int kpl = kpl_for(sh.K, sh.S);
    const int twm = twm_for(sh.Wo);
    a.TW = std::min(twm, sh.Wo);
    a.ctiles = (sh.Wo + a.TW - 1) / a.TW;
    a.bands = (sh.Ho + kWaves - 1) / kWaves;
    a.kgroups = (sh.K + kLanes * kpl - 1) / (kLanes * kpl);
    a.dec = dec;
    switch (sh.R) {
    case 1: return launch_reg_rs<1>(a, kpl, twm, s);
    case 3: return launch_reg_rs<3>(a, kpl, twm, s);
    default: return launch_reg_rs<5>(a, kpl, twm, s);
    }
}

}  // namespace isc
