// Weight-gradient kernel (declarations and, for the per-filter-size
// translation units that define ISC_DW_INSTANTIATE, the kernel and its
// launchers).
//
// Weight gradient with zero skipping, for training.  The paper measures the
// sparsity of rectified inputs during training (Sec. "Sparsity of ReLUs");
// the gradient of Eq. 1 with respect to the filter,
//   dw[k,c,r,s] = sum_{n,i,j} dy[n,k,i,j] * X^[n, c, i+r-P, j+s-P]   (stride 1),
// multiplies every input by output gradients, so a zero input contributes
// nothing and the work scales with the nonzeros as in ISC (Sec. "Sparse
// Convolution").  This is ISC step 2 with the roles of the filter and the
// output exchanged: a nonzero x at window row wy, shifted column xp meets the
// K-contiguous vector of output gradients dy[n, :, oy0 + wy - r, ox0 + xp - s]
// for every tap (r, s) whose output lies in the tile, and adds x times it to
// the K-contiguous gradient vector dw[:, c, r, s].
//
// A wavefront owns 64*KPL output maps (lanes over maps, as in the forward
// kernels), CH input channels and a contiguous range of output tiles (TH
// output rows, TW columns, one image each).  It keeps the CH*R*S*KPL
// gradient sums in registers for the whole range; per tile it loads the
// tile's output gradients for its maps (TH*TW*KPL registers) and, per channel,
// the input window that reaches the tile, takes a ballot of the zero test and
// scans it statically (tile::walk_scan_f): every set position runs a
// straight-line block of multiply-adds whose register indices are constants.
// The four wavefronts of a workgroup share maps and tile range and differ in
// channels: per tile they load the output gradients of their maps once,
// together, with consecutive lanes on consecutive columns of a map (whole
// cache lines), and transpose them through LDS so that each lane then reads
// its maps' values for every column.  Each wavefront finally stores its sums
// for its range; a second launch adds the ranges in order (deterministic, no
// atomics).
#pragma once

#include "sparse_tile.hpp"

namespace isc {
namespace dwk {

using tile::kLanes;
constexpr int kDwWaves = 4;
constexpr int kDwMinGroups = 1024;   // workgroups that fill 256 CUs four deep
constexpr int kDwMaxRegs = 100;      // gradient sums per lane, at most

struct DwArgs {
    const float *x;    // N x C x H x W
    const float *dy;   // N x K x Ho x Wo
    float *part;       // [splits][K][C*R*S]: sums of each tile range
    int N, C, H, W, K, P, Ho, Wo;
    int TWr, ctiles;   // output columns per tile in use, column tiles per row
    int bands;         // groups of TH output rows
    int cquads;        // groups of kDwWaves * CH channels
    int splits, per;   // tile ranges, tiles per range
    int ntiles;        // N * bands * ctiles
};

struct DwPlan {
    int kpl, th, ch, tw, TWr, ctiles, bands, kgroups, cquads, splits, per, ntiles;
};

// Channels per wavefront for a filter size and maps per lane: as many as
// kDwMaxRegs gradient sums allow, at most 16.
// Two-row tiles hold twice the output gradients: the channels are cut so
// that gradient sums and gradients together stay within the same budget.
constexpr int dw_ch_for(int RS, int KPL, int TH = 1) {
    const int room = kDwMaxRegs - (TH - 1) * 16 * KPL * 3 / 4;
    const int ch = room / (RS * RS * KPL);
    return ch < 1 ? 1 : (ch < 16 ? ch : 16);
}

// Launchers of the kernels of one filter size (sparse_dw_r{1,3,5}.hip).
hipError_t launch_r1(const DwArgs &a, const DwPlan &p, hipStream_t s);
hipError_t launch_r3(const DwArgs &a, const DwPlan &p, hipStream_t s);
hipError_t launch_r5(const DwArgs &a, const DwPlan &p, hipStream_t s);

}  // namespace dwk
}  // namespace isc

#ifdef ISC_DW_INSTANTIATE
namespace isc {
namespace dwk {
namespace {

template <int RS_, int KPL, int TH, int TW, int CH>
__global__ __launch_bounds__(kDwWaves * kLanes)
void sparse_dw_kernel(DwArgs a) {
    using T = tile::Shape<RS_, RS_, KPL, TH, TW>;
    constexpr int EPL = T::EPL, RS2 = RS_ * RS_;
    const int lane = threadIdx.x & (kLanes - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kLanes);
    int b = blockIdx.x;
    const int cq = b % a.cquads;
    b /= a.cquads;
    const int split = b % a.splits;
    const int kg = b / a.splits;
    const int cbase = (cq * kDwWaves + wave) * CH;
    const int kbase = kg * T::KW;
    const int C = a.C, H = a.H, W = a.W, K = a.K, P = a.P, Ho = a.Ho, Wo = a.Wo;
    const size_t HW = static_cast<size_t>(H) * W;

    float acc[CH][RS_][RS_][KPL];
#pragma unroll
    for (int ch = 0; ch < CH; ++ch)
#pragma unroll
        for (int r = 0; r < RS_; ++r)
#pragma unroll
            for (int s = 0; s < RS_; ++s)
#pragma unroll
                for (int j = 0; j < KPL; ++j) acc[ch][r][s][j] = 0.0f;

    // this lane's maps
    bool kok[KPL];
#pragma unroll
    for (int j = 0; j < KPL; ++j) kok[j] = kbase + lane * KPL + j < K;

    // the tile's output gradients, [row * TW + column][map] (pitch KW + 1);
    // the cooperative load: load i of the workgroup covers one row of 64 /
    // COLS maps, lane l column l % COLS of map l / COLS
    constexpr int KW = T::KW;
    constexpr int COLS = TW <= 16 ? 16 : 32;
    constexpr int MPI = kLanes / COLS;                 // maps per load
    constexpr int GPR = KW / MPI;                      // loads per tile row
    constexpr int NLD = TH * GPR / kDwWaves;           // loads per wavefront per tile
    static_assert((TH * GPR) % kDwWaves == 0, "cooperative load");
    static_assert(NLD <= 32, "validity bits");
    __shared__ float gs[2][TH * TW][KW + 1];
    const int lcol = lane % COLS;
    const int lmap = lane / COLS;

    // the loads of one tile, issued a tile ahead: its output gradients for
    // the cooperative load (vg: gs[hr * TW + ox][m] = dy[n, kbase + m,
    // oy0 + hr, ox0 + ox], zero past the map and past K) and this wavefront's channel
    // windows (vx, element e = q*64 + lane at window row wy = e / WCOLS,
    // input row oy0 - P + wy, shifted column xp, input column ox0 - P + xp;
    // inw: the element lies in the map and its column reaches the tile)
    float vg[NLD];
    uint32_t vok = 0;  // bit i: vg[i] is a gradient of the tile (else stored as zero)
    float vx[CH][EPL];
    bool inw[EPL];
    auto load_tile = [&](int t) {
        const int ct = t % a.ctiles;
        const int rest = t / a.ctiles;
        const int oy0 = (rest % a.bands) * TH;
        const int n = rest / a.bands;
        const int ox0 = ct * a.TWr;
        const int tw = min(a.TWr, Wo - ox0);
        // every load in bounds (clamped), the validity kept aside: a select
        // on the loaded value would let the compiler turn each load into a
        // branch with its own wait
        vok = 0;
#pragma unroll
        for (int i = 0; i < NLD; ++i) {
            const int li = wave * NLD + i;
            const int hr = li / GPR;
            const int m = (li - hr * GPR) * MPI + lmap;
            const int k = kbase + m;
            const int oy = oy0 + hr;
            const float *row =
                a.dy + ((static_cast<size_t>(n) * K + min(k, K - 1)) * Ho + min(oy, Ho - 1)) * Wo + ox0;
            vg[i] = row[min(lcol, tw - 1)];
            vok |= (k < K && lcol < tw && oy < Ho) ? (1u << i) : 0u;
        }
        int xoff[EPL];
#pragma unroll
        for (int q = 0; q < EPL; ++q) {
            const int e = q * kLanes + lane;
            const int wy = e / T::WCOLS;
            const int xp = e - wy * T::WCOLS;
            const int y = oy0 - P + wy, xx = ox0 - P + xp;
            inw[q] = e < T::WROWS * T::WCOLS && xp < tw + RS_ - 1 && y >= 0 && y < H && xx >= 0 && xx < W;
            xoff[q] = inw[q] ? y * W + xx : 0;
        }
        tile::static_for<0, CH>([&](auto chc) {
            constexpr int ch = decltype(chc)::value;
            const int c = min(cbase + ch, C - 1);
            const float *plane = a.x + (static_cast<size_t>(n) * C + c) * HW;
#pragma unroll
            for (int q = 0; q < EPL; ++q) vx[ch][q] = plane[xoff[q]];
        });
    };

    const int t0 = split * a.per;
    const int t1 = min(a.ntiles, t0 + a.per);
    if (t0 < t1) load_tile(t0);
#pragma unroll 1
    for (int t = t0; t < t1; ++t) {
        // the tile loaded last into LDS (one buffer of two: the other one is
        // still being read by wavefronts behind) and its windows into the
        // working registers, then the next tile's loads go out and land
        // while this one is scanned
        const int buf = (t - t0) & 1;
#pragma unroll
        for (int i = 0; i < NLD; ++i) {
            const int li = wave * NLD + i;
            const int hr = li / GPR;
            const int m = (li - hr * GPR) * MPI + lmap;
            if (lcol < TW) gs[buf][hr * TW + lcol][m] = ((vok >> i) & 1u) ? vg[i] : 0.0f;
        }
        // the windows move to working registers by explicit moves, which the
        // compiler cannot forward: the loaded registers are free again before
        // the next tile's loads, so none has to be copied (after a wait for
        // every load in flight) at the loop's back edge
        float cur[CH][EPL];
        bool inwin[EPL];
#pragma unroll
        for (int q = 0; q < EPL; ++q) inwin[q] = inw[q];
#pragma unroll
        for (int ch = 0; ch < CH; ++ch)
#pragma unroll
            for (int q = 0; q < EPL; ++q) asm volatile("v_mov_b32 %0, %1" : "=v"(cur[ch][q]) : "v"(vx[ch][q]));
        __syncthreads();
        if (t + 1 < t1) load_tile(t + 1);
        tile::Acc<T> g;
#pragma unroll
        for (int oy = 0; oy < TH; ++oy)
#pragma unroll
            for (int ox = 0; ox < TW; ++ox)
#pragma unroll
                for (int j = 0; j < KPL; ++j) g[oy][ox][j] = gs[buf][oy * TW + ox][lane * KPL + j];

        // per channel: ballot of the zero test, static scan of the window
        tile::static_for<0, CH>([&](auto chc) {
            constexpr int ch = decltype(chc)::value;
            if (cbase + ch < C) {  // wave-uniform
                unsigned long long mask[EPL];
#pragma unroll
                for (int q = 0; q < EPL; ++q)
                    mask[q] = __ballot(inwin[q] && (__float_as_uint(cur[ch][q]) & 0x7fffffffu) != 0u);
                // tap (r, s) reaches output (WY - r, XP - s) when it lies in
                // the tile
                auto blk = [&](auto wy_c, auto xp_c, float v) {
                    constexpr int WY = decltype(wy_c)::value, XP = decltype(xp_c)::value;
                    tile::static_for<0, RS_>([&](auto rc) {
                        constexpr int r = decltype(rc)::value, oy = WY - r;
                        if constexpr (oy >= 0 && oy < TH) {
                            tile::static_for<0, RS_>([&](auto sc) {
                                constexpr int sx = decltype(sc)::value, ox = XP - sx;
                                if constexpr (ox >= 0 && ox < TW) {
#pragma unroll
                                    for (int j = 0; j < KPL; ++j)
                                        acc[ch][r][sx][j] = __builtin_fmaf(v, g[oy][ox][j], acc[ch][r][sx][j]);
                                }
                            });
                        }
                    });
                };
                tile::walk_scan_f<T>(mask, cur[ch], blk);
            }
        });
    }

    // this range's sums: part[split][k][c][r][s]
    const size_t crs = static_cast<size_t>(C) * RS2;
    tile::static_for<0, CH>([&](auto chc) {
        constexpr int ch = decltype(chc)::value;
        const int c = cbase + ch;
        if (c < C) {
#pragma unroll
            for (int j = 0; j < KPL; ++j) {
                if (!kok[j]) continue;
                float *dst = a.part + (static_cast<size_t>(split) * K + kbase + lane * KPL + j) * crs +
                             static_cast<size_t>(c) * RS2;
#pragma unroll
                for (int r = 0; r < RS_; ++r)
#pragma unroll
                    for (int s = 0; s < RS_; ++s) dst[r * RS_ + s] = acc[ch][r][s][j];
            }
        }
    });
}

template <int RS_, int KPL, int TH, int TW>
hipError_t launch_dw_t(const DwArgs &a, const DwPlan &p, hipStream_t s) {
    constexpr int CH = dw_ch_for(RS_, KPL, TH);
    static_assert(CH >= 1 && CH * RS_ * RS_ * KPL <= kDwMaxRegs, "gradient sums");
    if (p.ch != CH) return hipErrorInvalidValue;
    const int64_t grid = static_cast<int64_t>(p.kgroups) * a.splits * a.cquads;
    sparse_dw_kernel<RS_, KPL, TH, TW, CH><<<static_cast<unsigned>(grid), kDwWaves * kLanes, 0, s>>>(a);
    return hipGetLastError();
}

// One-row tiles of 16 or 28 columns with 1, 2 or 4 maps per lane (four
// only with 16 columns); two-row tiles of 16 columns with 1 or 2.
template <int RS_>
hipError_t launch_dw_rs(const DwArgs &a, const DwPlan &p, hipStream_t s) {
    if (p.th == 2) {
        if (p.tw != 16) return hipErrorInvalidValue;
        return p.kpl == 1 ? launch_dw_t<RS_, 1, 2, 16>(a, p, s)
                          : (p.kpl == 2 ? launch_dw_t<RS_, 2, 2, 16>(a, p, s) : hipErrorInvalidValue);
    }
    switch (p.kpl) {
    case 1: return p.tw == 16 ? launch_dw_t<RS_, 1, 1, 16>(a, p, s) : launch_dw_t<RS_, 1, 1, 28>(a, p, s);
    case 2: return p.tw == 16 ? launch_dw_t<RS_, 2, 1, 16>(a, p, s) : launch_dw_t<RS_, 2, 1, 28>(a, p, s);
    default: return p.tw == 16 ? launch_dw_t<RS_, 4, 1, 16>(a, p, s) : hipErrorInvalidValue;
    }
}

}  // namespace
}  // namespace dwk
}  // namespace isc
#endif
