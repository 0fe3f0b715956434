// ISC steps 1-3 (Sec. "Sparse Convolution") in one launch, for stride-1
// convolutions with square 1x1, 3x3 or 5x5 filters, at most 64 output maps
// and a filter that fits in LDS (few input maps: LeNet conv2, an inception
// 5x5 branch).
//
// The paper builds each input map's nonzero list on the fly before using it.
// Here the list never leaves the wavefront: a wavefront loads the input rows
// its output tile needs straight from x (coalesced, one element per lane),
// takes a 64-bit ballot of the zero test per 64 elements, and walks the set
// bits in lane order -- row-major order, the paper's list order -- reading
// each nonzero's value and leaf key from its lane.  There are no compacted
// lists, row offsets or repacked filter in memory: the workgroup reads the
// filter once in its KCRS layout and transposes it into LDS (output map
// fastest, rows padded to 65 floats so that the transposing writes and the
// per-lane reads are free of bank conflicts).
//
// Work split and accumulation follow the filter-resident kernel: 16
// wavefronts per workgroup, wavefront w owns a TH x TW output tile (tile
// machinery in sparse_tile.hpp) of row group w / cs and takes the input
// channels c = (w mod cs) + i*cs; the cs partial tiles are summed through LDS
// in phase order and stored to NCHW (step 3).  Summation order per output is
// fixed for a given launch shape, so results are deterministic.
#include "sparse_tile.hpp"

#include <algorithm>
#include <cstdlib>

namespace isc {
namespace {

using tile::kLanes;
constexpr int kWaves = 16;
constexpr int kWPad = 65;  // LDS pitch of one filter tap's output maps
constexpr size_t kLdsMax = 160 * 1024;
constexpr int kFilterBatch = 8;   // filter elements a thread has in flight

struct FusedArgs {
    const float *x;  // N x C x H x W
    const float *w;  // K x C x R x S
    float *y;        // N x K x Ho x Wo
    int N, C, H, W, K, P, Ho, Wo;
    int cs;          // channel phases per row group
    int rg;          // row groups per workgroup (kWaves / cs)
    int bands;       // groups of rg * TH output rows
    int crs;         // C * R * S
    uint32_t m_crs;  // ceil(2^32 / crs), or 0 when crs == 1
    Decision dec;
};

__device__ __forceinline__ int div_crs(int e, int crs, uint32_t m) {
    return crs == 1 ? e : static_cast<int>(__umulhi(static_cast<uint32_t>(e), m));
}

template <int RS_, int TH, int TW>
__global__ __launch_bounds__(kWaves * kLanes)
void sparse_conv_fused_kernel(FusedArgs a) {
    using T = tile::Shape<RS_, RS_, 1, TH, TW>;
    constexpr int R = RS_, S = RS_, EPL = T::EPL;
    constexpr int NS = 4;                 // input-window register ring
    constexpr int TILEF = TH * TW * kLanes;

    extern __shared__ float lds[];  // filter [c*R*S + t][kWPad], later the phase tiles

    const int tid = threadIdx.x;
    const int lane = tid & (kLanes - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kLanes);
    const int cs = a.cs;
    const int phase = wave % cs;
    const int rgi = wave / cs;
    const int band = blockIdx.x % a.bands;
    const int n = blockIdx.x / a.bands;
    const int oy0 = (band * a.rg + rgi) * TH;
    const int C = a.C, H = a.H, W = a.W, P = a.P;
    const bool rows_ok = oy0 < a.Ho;
    // input rows of the tile's window, clipped to the map
    const int ylo = max(0, oy0 - P);
    const int yhi = min(H - 1, oy0 - P + T::WROWS - 1);
    const int nrows = rows_ok ? max(0, yhi - ylo + 1) : 0;
    const size_t HW = static_cast<size_t>(H) * W;
    const float *x_n = a.x + static_cast<size_t>(n) * C * HW;
    // this wavefront's channels: phase, phase + cs, ...
    const int ncw = phase < C ? (C - 1 - phase) / cs + 1 : 0;

    // lane l holds window element q*64 + l: its offset in the plane and its
    // leaf key (the same for every channel); lanes past the window read the
    // plane's first element and never count as nonzero
    int xoff[EPL], keyv[EPL];
    bool inwin[EPL];
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
        const int idx = q * kLanes + lane;
        inwin[q] = idx < nrows * W;
        const int dy = inwin[q] ? idx / W : 0;
        const int xx = inwin[q] ? idx - dy * W : 0;
        xoff[q] = inwin[q] ? (ylo + dy) * W + xx : 0;
        keyv[q] = (ylo + dy - (oy0 - P)) * T::WCOLS + xx + P;
    }

    // ring of NS register slots of input windows
    float xv[NS][EPL];
    auto issue = [&](auto slot_c, int i) {
        constexpr int SLOT = decltype(slot_c)::value;
        const int c = phase + min(i, ncw - 1) * cs;
        const float *plane = x_n + static_cast<size_t>(c) * HW;
#pragma unroll
        for (int q = 0; q < EPL; ++q) xv[SLOT][q] = plane[xoff[q]];
    };
    if (ncw > 0) tile::static_for<0, NS - 1>([&](auto sl) { issue(sl, decltype(sl)::value); });

    if (!decision_gate(a.dec, 1u)) return;

    // the filter, transposed into LDS: lds[t*kWPad + k] = w[k*CRS + t] for
    // t = c*R*S + r*S + s; coalesced reads along t, conflict-free writes
    {
        const int total = a.K * a.crs;
        for (int e0 = 0; e0 < total; e0 += kFilterBatch * kWaves * kLanes) {
            float tmp[kFilterBatch];
#pragma unroll
            for (int i = 0; i < kFilterBatch; ++i) {
                const int e = e0 + i * kWaves * kLanes + tid;
                tmp[i] = e < total ? a.w[e] : 0.0f;
            }
#pragma unroll
            for (int i = 0; i < kFilterBatch; ++i) {
                const int e = e0 + i * kWaves * kLanes + tid;
                if (e < total) {
                    const int k = div_crs(e, a.crs, a.m_crs);
                    const int t = e - k * a.crs;
                    lds[t * kWPad + k] = tmp[i];
                }
            }
        }
    }
    __syncthreads();

    tile::Acc<T> acc;
#pragma unroll
    for (int y = 0; y < TH; ++y)
#pragma unroll
        for (int x = 0; x < TW; ++x) acc[y][x][0] = 0.0f;

    // channels in order; the window NS-1 channels ahead is loaded before each
    // compute; the slot's values are copied to one set of registers so that
    // the walk (most of the code) is inlined once
    float cur[EPL];
#pragma unroll 1
    for (int i = 0; i < ncw; ++i) {
        tile::static_for<0, NS>([&](auto sl) {
            constexpr int B = decltype(sl)::value;
            if (i % NS == B) {
                if (i + NS - 1 < ncw) issue(std::integral_constant<int, (B + NS - 1) % NS>{}, i + NS - 1);
#pragma unroll
                for (int q = 0; q < EPL; ++q) cur[q] = xv[B][q];
            }
        });
        unsigned long long mask[EPL];
        bool any = false;
#pragma unroll
        for (int q = 0; q < EPL; ++q) {
            mask[q] = __ballot(inwin[q] && (__float_as_uint(cur[q]) & 0x7fffffffu) != 0u);
            any |= mask[q] != 0ull;
        }
        if (!any) continue;
        const int c = phase + i * cs;
        tile::Wts<T> w;
        tile::load_weights<T>(lds + static_cast<size_t>(c) * R * S * kWPad, lane, w, kWPad);
        tile::wait_lgkm0();
        // one copy of the walk: the q-th mask, keys and values by selects
#pragma unroll 1
        for (int q = 0; q < EPL; ++q) {
            unsigned long long m = mask[0];
            int kv = keyv[0], vb = __float_as_int(cur[0]);
#pragma unroll
            for (int u = 1; u < EPL; ++u)
                if (q == u) {
                    m = mask[u];
                    kv = keyv[u];
                    vb = __float_as_int(cur[u]);
                }
            tile::walk_mask<T>(m, kv, vb, acc, w);
        }
    }

    const size_t plane_out = static_cast<size_t>(a.Ho) * a.Wo;
    float *yrow = a.y + static_cast<size_t>(n) * a.K * plane_out + static_cast<size_t>(oy0) * a.Wo;
    if (cs == 1) {
        if (rows_ok) tile::store_tile<T>(acc, yrow, plane_out, a.Wo, 0, lane, a.K, a.Ho - oy0, a.Wo);
        return;
    }
    // the cs phase tiles of a row group are summed through LDS (the filter is
    // no longer needed): every wavefront writes its tile, then sums the tile
    // positions p = phase (mod cs) over the phases in phase order and stores
    // them (step 3)
    __syncthreads();
    float *red = lds;  // [waves][TH*TW][64]
#pragma unroll
    for (int y = 0; y < TH; ++y)
#pragma unroll
        for (int x = 0; x < TW; ++x) red[(static_cast<size_t>(wave) * TH * TW + y * TW + x) * kLanes + lane] = acc[y][x][0];
    __syncthreads();
    if (!rows_ok || lane >= a.K) return;
    const float *grp = red + static_cast<size_t>(rgi) * cs * TILEF + lane;
#pragma unroll 2
    for (int pos = phase; pos < TH * TW; pos += cs) {
        const int oy = pos / TW, ox = pos - (pos / TW) * TW;
        if (oy0 + oy >= a.Ho || ox >= a.Wo) continue;
        const float *src = grp + static_cast<size_t>(pos) * kLanes;
        float part[kWaves];
#pragma unroll
        for (int p = 0; p < kWaves; ++p) part[p] = p < cs ? src[static_cast<size_t>(p) * TILEF] : 0.0f;
        float sum = part[0];
#pragma unroll
        for (int p = 1; p < kWaves; ++p)
            if (p < cs) sum += part[p];
        yrow[static_cast<size_t>(lane) * plane_out + oy * a.Wo + ox] = sum;
    }
}

struct FusedPlan {
    int th, tw, cs;
    size_t lds;
};

int fused_tw(int Wo) { return Wo <= 8 ? 8 : (Wo <= 16 ? 16 : 28); }

size_t fused_lds(const SparseShape &sh, int th, int tw, int cs) {
    const size_t filt = static_cast<size_t>(sh.C) * sh.R * sh.S * kWPad;
    const size_t tiles = cs > 1 ? static_cast<size_t>(kWaves) * th * tw * kLanes : 0;
    return sizeof(float) * std::max(filt, tiles);
}

constexpr int kMaxTile = 32;  // accumulators per lane
constexpr int kMinGroups = 256;  // workgroups that fill the CUs once

constexpr int max_tile(int) { return kMaxTile; }

// Tallest tile (up to max_tile accumulators per lane), then the fewest
// channel phases whose row groups still fit the output height, within LDS;
// a plan with fewer than kMinGroups workgroups is kept only if no other fits.
// ISC_FUSED_TH caps the tile height (for measurements).
bool fused_plan(const SparseShape &sh, FusedPlan *plan) {
    if (sh.T != 1 || sh.R != sh.S || !(sh.R == 1 || sh.R == 3 || sh.R == 5)) return false;
    if (sh.Wo > 28 || sh.K > kLanes) return false;
    if (static_cast<int64_t>(sh.K) * sh.C * sh.R * sh.S >= (int64_t(1) << 30)) return false;
    const int tw = fused_tw(sh.Wo);
    int th_cap = 8;
    if (const char *env = std::getenv("ISC_FUSED_TH")) th_cap = std::max(1, std::atoi(env));
    bool found = false;
    for (int th : {8, 4, 2, 1}) {
        if (th * tw > max_tile(sh.R) || th > th_cap) continue;
        const int rows_need = (sh.Ho + th - 1) / th;
        for (int cs = 1; cs <= kWaves; cs *= 2) {
            const int rg = kWaves / cs;
            if (rg > rows_need && cs < kWaves && cs * 2 <= sh.C) continue;  // more phases: fewer idle rows
            if (cs > sh.C) break;
            const size_t lds = fused_lds(sh, th, tw, cs);
            if (lds > kLdsMax) continue;
            const int64_t groups = static_cast<int64_t>(sh.N) * ((sh.Ho + rg * th - 1) / (rg * th));
            if (!found || groups >= kMinGroups) {
                *plan = FusedPlan{th, tw, cs, lds};
                found = true;
            }
            if (groups >= kMinGroups) return true;
            break;
        }
    }
    return found;
}

template <int RS_, int TH, int TW>
hipError_t launch_fused_t(const FusedArgs &a, size_t lds, hipStream_t s) {
    if constexpr (TH * TW > max_tile(RS_)) {
        return hipErrorInvalidValue;
    } else {
        auto kern = sparse_conv_fused_kernel<RS_, TH, TW>;
        if (lds > 64 * 1024) {
            hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
            if (e != hipSuccess) return e;
        }
        kern<<<a.N * a.bands, kWaves * kLanes, lds, s>>>(a);
        return hipGetLastError();
    }
}

template <int RS_, int TW>
hipError_t launch_fused_th(const FusedArgs &a, int th, size_t lds, hipStream_t s) {
    switch (th) {
    case 8: return launch_fused_t<RS_, 8, TW>(a, lds, s);
    case 4: return launch_fused_t<RS_, 4, TW>(a, lds, s);
    case 2: return launch_fused_t<RS_, 2, TW>(a, lds, s);
    default: return launch_fused_t<RS_, 1, TW>(a, lds, s);
    }
}

template <int RS_>
hipError_t launch_fused_rs(const FusedArgs &a, const FusedPlan &p, hipStream_t s) {
    switch (p.tw) {
    case 8: return launch_fused_th<RS_, 8>(a, p.th, p.lds, s);
    case 16: return launch_fused_th<RS_, 16>(a, p.th, p.lds, s);
    default: return launch_fused_th<RS_, 28>(a, p.th, p.lds, s);
    }
}

}  // namespace

bool sparse_fused_applies(const SparseShape &sh) {
    FusedPlan p;
    return fused_plan(sh, &p);
}

hipError_t launch_sparse_fused(const SparseShape &sh, const float *x, const float *w, float *y, const Decision &dec,
                               hipStream_t s) {
    FusedPlan p;
    if (!fused_plan(sh, &p)) return hipErrorInvalidValue;
    if (const char *env = std::getenv("ISC_FUSED_CS")) {  // tuning override
        const int v = std::atoi(env);
        if (v >= 1 && v <= kWaves && kWaves % v == 0 && v <= sh.C) {
            const size_t lds = fused_lds(sh, p.th, p.tw, v);
            if (lds <= kLdsMax) {
                p.cs = v;
                p.lds = lds;
            }
        }
    }
    FusedArgs a{};
    a.x = x;
    a.w = w;
    a.y = y;
    a.N = sh.N; a.C = sh.C; a.H = sh.H; a.W = sh.W; a.K = sh.K; a.P = sh.P; a.Ho = sh.Ho; a.Wo = sh.Wo;
    a.cs = p.cs;
    a.rg = kWaves / p.cs;
    a.bands = (sh.Ho + a.rg * p.th - 1) / (a.rg * p.th);
    a.crs = sh.C * sh.R * sh.S;
    a.m_crs = a.crs <= 1 ? 0u : static_cast<uint32_t>((0x100000000ull + a.crs - 1) / a.crs);
    a.dec = dec;
    switch (sh.R) {
    case 1: return launch_fused_rs<1>(a, p, s);
    case 3: return launch_fused_rs<3>(a, p, s);
    default: return launch_fused_rs<5>(a, p, s);
    }
}

}  // namespace isc
