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
// kernels), CH input channels and a contiguous range of output tiles (one
// output row, TW columns, one image each).  It keeps the CH*R*S*KPL
// gradient sums in registers for the whole range; per tile it loads the
// tile's output gradients for its maps (TW*KPL registers) and, per channel,
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
    int cquads;        // groups of kDwWaves * CH channels
    int splits, per;   // tile ranges, tiles per range
    int ntiles;        // N * Ho * ctiles
};

struct DwPlan {
    int kpl, ch, tw, TWr, ctiles, kgroups, cquads, splits, per, ntiles;
};

// Channels per wavefront for a filter size and maps per lane: as many as
// kDwMaxRegs gradient sums allow, at most 16.
constexpr int dw_ch_for(int RS, int KPL) {
    return kDwMaxRegs / (RS * RS * KPL) < 16 ? kDwMaxRegs / (RS * RS * KPL) : 16;
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

template <int RS_, int KPL, int TW, int CH>
__global__ __launch_bounds__(kDwWaves * kLanes)
void sparse_dw_kernel(DwArgs a) {
    using T = tile::Shape<RS_, RS_, KPL, 1, TW>;
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

    // the tile's output gradients, [column][map] (pitch KW + 1); the
    // cooperative load: lane l of a load covers column l % COLS of map
    // l / COLS of a group of 64 / COLS maps
    constexpr int KW = T::KW;
    constexpr int COLS = TW <= 16 ? 16 : 32;
    constexpr int MPI = kLanes / COLS;                 // maps per load
    constexpr int NLD = KW / (MPI * kDwWaves);         // loads per wavefront per tile
    static_assert(KW % (MPI * kDwWaves) == 0, "cooperative load");
    static_assert(NLD <= 32, "validity bits");
    __shared__ float gs[2][TW][KW + 1];
    const int lcol = lane % COLS;
    const int lmap = lane / COLS;

    // the loads of one tile, issued a tile ahead: its output gradients for
    // the cooperative load (vg: gs[ox][m] = dy[n, kbase + m, oy0, ox0 + ox],
    // zero past the map's columns and past K) and this wavefront's channel
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
        const int oy0 = rest % Ho;
        const int n = rest / Ho;
        const int ox0 = ct * a.TWr;
        const int tw = min(a.TWr, Wo - ox0);
        // every load in bounds (clamped), the validity kept aside: a select
        // on the loaded value would let the compiler turn each load into a
        // branch with its own wait
        vok = 0;
#pragma unroll
        for (int i = 0; i < NLD; ++i) {
            const int m = (wave * NLD + i) * MPI + lmap;
            const int k = kbase + m;
            const float *row = a.dy + ((static_cast<size_t>(n) * K + min(k, K - 1)) * Ho + oy0) * Wo + ox0;
            vg[i] = row[min(lcol, tw - 1)];
            vok |= (k < K && lcol < tw) ? (1u << i) : 0u;
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
            const int m = (wave * NLD + i) * MPI + lmap;
            if (lcol < TW) gs[buf][lcol][m] = ((vok >> i) & 1u) ? vg[i] : 0.0f;
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
        for (int ox = 0; ox < TW; ++ox)
#pragma unroll
            for (int j = 0; j < KPL; ++j) g[0][ox][j] = gs[buf][ox][lane * KPL + j];

        // per channel: ballot of the zero test, static scan of the window
        tile::static_for<0, CH>([&](auto chc) {
            constexpr int ch = decltype(chc)::value;
            if (cbase + ch < C) {  // wave-uniform
                unsigned long long mask[EPL];
#pragma unroll
                for (int q = 0; q < EPL; ++q)
                    mask[q] = __ballot(inwin[q] && (__float_as_uint(cur[ch][q]) & 0x7fffffffu) != 0u);
                // one output row: the tap row is r = WY; the tap column s
                // reaches output column XP - s when it lies in the tile
                auto blk = [&](auto wy_c, auto xp_c, float v) {
                    constexpr int WY = decltype(wy_c)::value, XP = decltype(xp_c)::value;
                    tile::static_for<0, RS_>([&](auto sc) {
                        constexpr int sx = decltype(sc)::value, ox = XP - sx;
                        if constexpr (ox >= 0 && ox < TW) {
#pragma unroll
                            for (int j = 0; j < KPL; ++j)
                                acc[ch][WY][sx][j] = __builtin_fmaf(v, g[0][ox][j], acc[ch][WY][sx][j]);
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

template <int RS_, int KPL, int TW>
hipError_t launch_dw_t(const DwArgs &a, int kgroups, hipStream_t s) {
    constexpr int CH = dw_ch_for(RS_, KPL);
    static_assert(CH >= 1 && CH * RS_ * RS_ * KPL <= kDwMaxRegs, "gradient sums");
    const int64_t grid = static_cast<int64_t>(kgroups) * a.splits * a.cquads;
    sparse_dw_kernel<RS_, KPL, TW, CH><<<static_cast<unsigned>(grid), kDwWaves * kLanes, 0, s>>>(a);
    return hipGetLastError();
}

// 16- or 28-column tiles; four maps per lane only with 16-column tiles.
template <int RS_>
hipError_t launch_dw_rs(const DwArgs &a, const DwPlan &p, hipStream_t s) {
    switch (p.kpl) {
    case 1: return p.tw == 16 ? launch_dw_t<RS_, 1, 16>(a, p.kgroups, s) : launch_dw_t<RS_, 1, 28>(a, p.kgroups, s);
    case 2: return p.tw == 16 ? launch_dw_t<RS_, 2, 16>(a, p.kgroups, s) : launch_dw_t<RS_, 2, 28>(a, p.kgroups, s);
    default: return p.tw == 16 ? launch_dw_t<RS_, 4, 16>(a, p.kgroups, s) : hipErrorInvalidValue;
    }
}

}  // namespace
}  // namespace dwk
}  // namespace isc
#endif
