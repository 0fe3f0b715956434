// ISC steps 2 and 3 (Sec. "Sparse Convolution"), register-tile kernel with
// the whole filter resident in LDS: stride 1, square 1x1, 3x3 and 5x5
// filters whose weights for 64 output maps fit in LDS (few input maps, e.g.
// LeNet conv2 or an inception 5x5 branch).
//
// Small layers have too few output rows to fill the GPU with one wavefront
// per row, and per-channel barriers would then dominate.  Here a workgroup of
// 16 wavefronts loads all C channels' weights of its 64*KPL output maps into
// LDS once (direct global -> LDS loads), after which every wavefront runs
// without barriers.  Wavefront w owns the output tile of TH rows x TW columns
// (tile machinery in sparse_tile.hpp) of row group w / cs and takes the input
// channels c = (w mod cs) + i*cs ("phase" w mod cs); its nonzero runs come
// from the compacted lists through a four-slot register pipeline.  The cs
// phase tiles of a row group are then added through LDS in phase order, and
// phase 0 stores the sum to NCHW (step 3).  Summation order per output is
// fixed for a given launch shape, so results are deterministic.
#include "sparse_tile.hpp"

#include <algorithm>
#include <cstdlib>

namespace isc {
namespace {

using tile::kLanes;
constexpr int kWaves = 16;
constexpr size_t kLdsMax = 160 * 1024;

struct ResArgs {
    const int32_t *row_ptr;
    const NzEntry *nz;
    const float *wt;  // [C][R][S][Kp], K contiguous
    float *y;
    int N, C, H, W, K, Kp, P, Ho, Wo;
    int cs;       // channel phases per row group
    int rg;       // row groups per workgroup (kWaves / cs)
    int bands;    // groups of rg * TH output rows
    int kgroups;  // groups of 64 * KPL output maps
    int cpw;      // channel slots per wavefront in the offsets table: ceil(C / cs)
    int wfloats;  // LDS floats of the weights, whole 256-float blocks
    int lfloats;  // LDS floats before the offsets: weights, or the phase tiles if larger
    Decision dec;
};

template <int RS_, int KPL, int TH, int TW>
__global__ __launch_bounds__(kWaves * kLanes)
void sparse_conv_res_kernel(ResArgs a) {
    using T = tile::Shape<RS_, RS_, KPL, TH, TW>;
    constexpr int R = RS_, S = RS_, KW = T::KW, EPL = T::EPL;
    constexpr int CHF = R * S * KW;     // floats of one channel
    constexpr int NOFF = T::WROWS + 1;  // row offsets kept per channel
    constexpr int TILEF = TH * TW * KW;  // floats of one wavefront's tile
    constexpr int NS = 4;                // run ring slots

    extern __shared__ float4 lds4[];
    float *wlds = reinterpret_cast<float *>(lds4);                     // [C][R*S][KW]
    int32_t *offs_all = reinterpret_cast<int32_t *>(wlds + a.lfloats);  // [waves][cpw][NOFF]

    const int lane = threadIdx.x & (kLanes - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kLanes);
    const int cs = a.cs;
    const int phase = wave % cs;
    const int rgi = wave / cs;
    int b = blockIdx.x;
    const int kg = b % a.kgroups;
    b /= a.kgroups;
    const int band = b % a.bands;
    const int n = b / a.bands;
    const int oy0 = (band * a.rg + rgi) * TH;
    const int kbase = kg * KW;
    const int C = a.C, H = a.H, W = a.W, P = a.P, Kp = a.Kp;
    const bool rows_ok = oy0 < a.Ho;
    // input rows of the tile's window, clipped to the map
    const int ylo = max(0, oy0 - P);
    const int yhi = min(H - 1, oy0 - P + T::WROWS - 1);
    const int nrows = rows_ok ? max(0, yhi - ylo + 1) : 0;
    const size_t HW = static_cast<size_t>(H) * W;
    const NzEntry *nz_n = a.nz + static_cast<size_t>(n) * C * HW;
    // this wavefront's channels: phase, phase + cs, ...
    const int ncw = phase < C ? (C - 1 - phase) / cs + 1 : 0;
    int32_t *offs = offs_all + wave * a.cpw * NOFF;

    // 1. row offsets of the window rows of this wavefront's channels (at most
    // 2 * 64 values, loaded before the decision so that both loads are in
    // flight together), then to LDS
    int32_t offv[2];
    {
        const int32_t *rp_n = a.row_ptr + static_cast<size_t>(n) * C * (H + 1);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int idx = lane + h * kLanes;
            const int i = idx / NOFF;
            const int j = idx - i * NOFF;
            const int c = min(phase + i * cs, C - 1);
            const bool use = idx < ncw * NOFF && j <= nrows && nrows > 0;
            offv[h] = use ? rp_n[static_cast<size_t>(c) * (H + 1) + min(ylo + j, H)] : 0;
        }
    }
    if (!decision_gate(a.dec, 1u)) return;
#pragma unroll
    for (int h = 0; h < 2; ++h)
        if (lane + h * kLanes < ncw * NOFF) offs[lane + h * kLanes] = offv[h];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // ring of NS register slots of nonzero runs; lanes past a run re-read
    // its last entry, an empty run reads the slot it would start at (in
    // bounds thanks to the list's 256-entry tail)
    NzEntry run[NS][EPL];
    auto issue = [&](auto slot_c, int i) {
        constexpr int SLOT = decltype(slot_c)::value;
        const int ii = min(i, ncw - 1);
        const int c = phase + ii * cs;
        const int e0 = __builtin_amdgcn_readfirstlane(offs[ii * NOFF]);
        const int last = max(__builtin_amdgcn_readfirstlane(offs[ii * NOFF + nrows]) - e0 - 1, 0);
        const NzEntry *src = nz_n + static_cast<size_t>(c) * HW + e0;
#pragma unroll
        for (int q = 0; q < EPL; ++q) run[SLOT][q] = src[min(q * kLanes + lane, last)];
    };

    // 2. the runs of the first NS-1 channels and every channel's weights of
    // this map group (global -> LDS; lanes past the last whole chunk re-read
    // it into the padding) in flight together
    if (ncw > 0) tile::static_for<0, NS - 1>([&](auto sl) { issue(sl, decltype(sl)::value); });
    {
        const int total = C * CHF;
        const int blocks = a.wfloats / 256;
        for (int d = wave; d < blocks; d += kWaves) {
            const int g = min(d * 256 + lane * 4, total - 4);
            const int c = g / CHF;
            const int rem = g - c * CHF;
            const int tap = rem / KW;
            const int koff = rem - tap * KW;
            const float *src = a.wt + (static_cast<size_t>(c) * R * S + tap) * Kp + min(kbase + koff, Kp - 4);
            tile::load_lds16(src, &lds4[d * kLanes]);
        }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    tile::Acc<T> acc;
#pragma unroll
    for (int y = 0; y < TH; ++y)
#pragma unroll
        for (int x = 0; x < TW; ++x)
#pragma unroll
            for (int j = 0; j < KPL; ++j) acc[y][x][j] = 0.0f;

    // 3. channels in order; the run NS-1 channels ahead is issued before each
    // compute, and the wait leaves exactly those loads in flight.  The slot's
    // run is copied to one set of registers so that the walk (most of the
    // code) is inlined once.
    NzEntry cur[EPL];
#pragma unroll 1
    for (int i = 0; i < ncw; ++i) {
        const bool ahead = i + NS - 1 < ncw;
        tile::static_for<0, NS>([&](auto sl) {
            constexpr int B = decltype(sl)::value;
            if (i % NS == B) {
                if (ahead) {
                    issue(std::integral_constant<int, (B + NS - 1) % NS>{}, i + NS - 1);
                    tile::wait_vm<(NS - 1) * EPL, false>();
                } else {
                    // tail: channels i+1 .. ncw-1 may stay in flight
                    switch (ncw - 1 - i) {
                    case 0: tile::wait_vm<0, false>(); break;
                    case 1: tile::wait_vm<EPL, false>(); break;
                    default: tile::wait_vm<2 * EPL, false>(); break;
                    }
                }
#pragma unroll
                for (int q = 0; q < EPL; ++q) cur[q] = run[B][q];
            }
        });
        const int c = phase + i * cs;
        const int e0 = __builtin_amdgcn_readfirstlane(offs[i * NOFF]);
        const int len = __builtin_amdgcn_readfirstlane(offs[i * NOFF + nrows]) - e0;
        if (len > 0) {
            tile::Wts<T> w;
            tile::load_weights<T>(wlds + c * CHF, lane, w);
            tile::wait_lgkm0();
            // the tile spans the whole output width: every column is in the window
            tile::walk<T, false>(cur, len, oy0 - P, P, 0, W - 1, acc, w);
        }
    }
    __builtin_amdgcn_s_waitcnt(0);

    const size_t plane_out = static_cast<size_t>(a.Ho) * a.Wo;
    float *yrow = a.y + static_cast<size_t>(n) * a.K * plane_out + static_cast<size_t>(oy0) * a.Wo;
    if (cs == 1) {
        // step 3: each lane stores its accumulators to NCHW
        if (rows_ok) tile::store_tile<T>(acc, yrow, plane_out, a.Wo, kbase, lane, a.K, a.Ho - oy0, a.Wo);
        return;
    }
    // the cs phase tiles of a row group are summed through LDS (the weights
    // are no longer needed): every wavefront writes its tile, then sums the
    // tile positions p = phase (mod cs) over the phases in phase order and
    // stores them (step 3)
    __syncthreads();
    float *red = wlds;  // [waves][TH*TW][KW]
#pragma unroll
    for (int y = 0; y < TH; ++y)
#pragma unroll
        for (int x = 0; x < TW; ++x)
#pragma unroll
            for (int j = 0; j < KPL; ++j)
                red[(static_cast<size_t>(wave) * TH * TW + y * TW + x) * KW + lane * KPL + j] = acc[y][x][j];
    __syncthreads();
    if (!rows_ok) return;
    const float *grp = red + static_cast<size_t>(rgi) * cs * TILEF;
#pragma unroll 2
    for (int pos = phase; pos < TH * TW; pos += cs) {
        const int oy = pos / TW, ox = pos - (pos / TW) * TW;
        if (oy0 + oy >= a.Ho || ox >= a.Wo) continue;
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
            const int k = kbase + lane * KPL + j;
            const float *src = grp + static_cast<size_t>(pos) * KW + lane * KPL + j;
            float part[kWaves];
#pragma unroll
            for (int p = 0; p < kWaves; ++p) part[p] = p < cs ? src[static_cast<size_t>(p) * TILEF] : 0.0f;
            float sum = part[0];
#pragma unroll
            for (int p = 1; p < kWaves; ++p)
                if (p < cs) sum += part[p];
            if (k < a.K) yrow[static_cast<size_t>(k) * plane_out + oy * a.Wo + ox] = sum;
        }
    }
}

struct ResPlan {
    int th, tw, cs, kpl;
    size_t lfloats;  // weights, or the phase tiles when larger
    size_t lds;      // bytes: lfloats, then the offsets table
};

int res_tw(int Wo) { return Wo <= 8 ? 8 : (Wo <= 16 ? 16 : 28); }

size_t res_wfloats(int C, int RS, int kpl) {
    const size_t f = static_cast<size_t>(C) * RS * RS * kLanes * kpl;
    return (f + 255) / 256 * 256;
}

// LDS of a launch shape: the weights (reused for the phase tiles when cs >
// 1), then the offsets table.
void res_lds(const SparseShape &sh, ResPlan *p) {
    const size_t wf = res_wfloats(sh.C, sh.R, p->kpl);
    const size_t tiles = p->cs > 1 ? static_cast<size_t>(kWaves) * p->th * p->tw * kLanes * p->kpl : 0;
    p->lfloats = std::max(wf, tiles);
    const size_t cpw = (sh.C + p->cs - 1) / p->cs;
    p->lds = p->lfloats * sizeof(float) + sizeof(int32_t) * kWaves * cpw * (p->th + sh.R);
}

// Row offsets one wavefront keeps: its channels times (window rows + 1).
int res_offsets(const SparseShape &sh, const ResPlan &p) { return (sh.C + p.cs - 1) / p.cs * (p.th + sh.R); }

// Choose the tile height and the channel phases: the tallest tile (up to
// 32 accumulators per lane), then the fewest phases whose row groups still
// fit the output height, within LDS.
bool res_plan(const SparseShape &sh, ResPlan *plan) {
    if (sh.T != 1 || sh.R != sh.S || !(sh.R == 1 || sh.R == 3 || sh.R == 5)) return false;
    if (sh.Wo > 28 || sh.K > kLanes) return false;  // one column tile, KPL = 1
    const int tw = res_tw(sh.Wo);
    const int kpl = 1;
    const int ths[] = {4, 2, 1};
    for (int th : ths) {
        if (th * tw > 32) continue;
        // the window of th rows must stage in the run registers (always true
        // when the tile spans the width: W <= TW + S - 1)
        const int rows_need = (sh.Ho + th - 1) / th;  // row groups the image needs
        for (int cs = 1; cs <= kWaves; cs *= 2) {
            const int rg = kWaves / cs;
            if (rg > rows_need && cs < kWaves && cs * 2 <= sh.C) continue;  // more phases: fewer idle rows
            if (cs > sh.C) break;
            ResPlan p{th, tw, cs, kpl, 0, 0};
            res_lds(sh, &p);
            if (p.lds > kLdsMax || res_offsets(sh, p) > 2 * kLanes) continue;
            *plan = p;
            return true;
        }
    }
    return false;
}

template <int RS_, int TH, int TW>
hipError_t launch_res_t(const ResArgs &a, size_t lds, hipStream_t s) {
    if constexpr (TH * TW > 32) {
        return hipErrorInvalidValue;
    } else {
        auto kern = sparse_conv_res_kernel<RS_, 1, TH, TW>;
        if (lds > 64 * 1024) {
            hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
            if (e != hipSuccess) return e;
        }
        const int grid = a.N * a.bands * a.kgroups;
        kern<<<grid, kWaves * kLanes, lds, s>>>(a);
        return hipGetLastError();
    }
}

template <int RS_, int TW>
hipError_t launch_res_th(const ResArgs &a, int th, size_t lds, hipStream_t s) {
    switch (th) {
    case 4: return launch_res_t<RS_, 4, TW>(a, lds, s);
    case 2: return launch_res_t<RS_, 2, TW>(a, lds, s);
    default: return launch_res_t<RS_, 1, TW>(a, lds, s);
    }
}

template <int RS_>
hipError_t launch_res_rs(const ResArgs &a, const ResPlan &p, hipStream_t s) {
    switch (p.tw) {
    case 8: return launch_res_th<RS_, 8>(a, p.th, p.lds, s);
    case 16: return launch_res_th<RS_, 16>(a, p.th, p.lds, s);
    default: return launch_res_th<RS_, 28>(a, p.th, p.lds, s);
    }
}

}  // namespace

bool sparse_res_applies(const SparseShape &sh) {
    ResPlan p;
    return res_plan(sh, &p);
}

hipError_t launch_sparse_res(const SparseShape &sh, const int32_t *row_ptr, const NzEntry *nz, const float *wt,
                             float *y, const Decision &dec, hipStream_t s) {
    ResPlan p;
    if (!res_plan(sh, &p)) return hipErrorInvalidValue;
    if (sh.tu.phases > 0) {  // a caller's override
        const int v = sh.tu.phases;
        ResPlan q = p;
        q.cs = v;
        if (v >= 1 && v <= kWaves && kWaves % v == 0 && v <= sh.C) {
            res_lds(sh, &q);
            if (q.lds <= kLdsMax && res_offsets(sh, q) <= 2 * kLanes) p = q;
        }
    }
    ResArgs a{};
    a.row_ptr = row_ptr;
    a.nz = nz;
    a.wt = wt;
    a.y = y;
    a.N = sh.N; a.C = sh.C; a.H = sh.H; a.W = sh.W; a.K = sh.K;
    a.Kp = (sh.K + kLanes - 1) / kLanes * kLanes;
    a.P = sh.P; a.Ho = sh.Ho; a.Wo = sh.Wo;
    a.cs = p.cs;
    a.rg = kWaves / p.cs;
    a.bands = (sh.Ho + a.rg * p.th - 1) / (a.rg * p.th);
    a.kgroups = (sh.K + kLanes * p.kpl - 1) / (kLanes * p.kpl);
    a.cpw = (sh.C + p.cs - 1) / p.cs;
    a.wfloats = static_cast<int>(res_wfloats(sh.C, sh.R, p.kpl));
    a.lfloats = static_cast<int>(p.lfloats);
    a.dec = dec;
    if (p.lds > kLdsMax) return hipErrorInvalidValue;
    switch (sh.R) {
    case 1: return launch_res_rs<1>(a, p, s);
    case 3: return launch_res_rs<3>(a, p, s);
    default: return launch_res_rs<5>(a, p, s);
    }
}

}  // namespace isc
