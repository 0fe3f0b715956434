// Filter-ring kernel (declarations and, for the per-filter-size translation
// units that define ISC_FRING_INSTANTIATE, the kernel and its launchers).
//
// ISC steps 1-3 (Sec. "Sparse Convolution") in one launch for stride-1
// convolutions with square 1x1, 3x3 or 5x5 filters whose filter does not fit
// in LDS (many input or output maps: AlexNet conv2-5, an inception 3x3
// branch): the input is compacted on the fly as in the filter-resident kernel
// (sparse_fused.hip), and the filter is streamed through LDS.
//
// The output of every image is cut into TH x TW tiles, numbered image by
// image, row band by row band; wavefront w of workgroup b owns tile 4b + w
// (any image: the four wavefronts share only the channel's weights), with
// 64*KPL output maps in registers (tile machinery in sparse_tile.hpp).  The
// flat tile list leaves no wavefront idle on a ragged last band, except in
// the launch's last workgroup.  Input channels go in order through a ring
// of NBUF stages: stage c holds channel c's R*S*64*KPL weights (from the
// K-contiguous repacked filter) and each wavefront's input window of the
// channel -- (TH+R-1) rows x (TW+S-1) columns in leaf-key order, padding
// read as zero -- all brought in by direct global->LDS loads.  No register
// is the target of a load in flight, so the only waits are the kernel's own:
// stages are issued NBUF-1 channels ahead and each channel waits for exactly
// the stage it consumes, then one barrier.  Per channel a
// wavefront reads the weights into registers, takes a ballot of the zero test
// over its window and scans the window statically (walk_scan): every set
// position runs the straight-line block of its (row, column).  Each lane
// finally stores its accumulators to NCHW (step 3).  Summation order per
// output is fixed (channels in order, window order within a channel), so
// results are deterministic.
#pragma once

#include "sparse_tile.hpp"

namespace isc {
namespace fring {

using tile::kLanes;
constexpr size_t kLdsMax = 160 * 1024;

struct FringArgs {
    const float *x;   // N x C x H x W
    const float *wt;  // [C][R][S][Kp], K contiguous, zero past K
    float *y;         // N x K x Ho x Wo
    int N, C, H, W, K, Kp, P, Ho, Wo;
    int ctiles;       // column tiles per row band, ceil(Wo / TW)
    int rtiles;       // row bands per image, ceil(Ho / TH)
    int ntiles;       // N * rtiles * ctiles
    int kgroups;      // groups of 64 * KPL output maps
    Decision dec;
    Epilogue epi;     // rectifier and census of y
};

// A register tile: KPL maps per lane, TH x TW outputs, so TH * TW * KPL
// accumulators and R*S*KPL weights per lane; NW wavefronts per workgroup
// share each stage of the ring (4: two workgroups per CU, each with half
// of the LDS; 8: one workgroup per CU with all of it, so a deeper ring and
// half the weight traffic per wavefront).
struct TileChoice {
    int kpl, th, tw, nw;
};

constexpr int kMaxAcc = 160;      // accumulators per lane
constexpr int kMaxRegs = 216;     // accumulators + weights per lane

constexpr bool fring_fits(int RS, int KPL, int TH, int TW) {
    return TH * TW * KPL <= kMaxAcc && TH * TW * KPL + RS * RS * KPL <= kMaxRegs;
}

// The tiles compiled for each filter size, the choice's candidates.  Tall
// tiles feed every scanned nonzero to more outputs (R x S filters: up to
// TH*TW*R*S / ((TH+R-1)(TW+S-1)) taps, times KPL maps per lane), which is
// what the scan's scalar work per nonzero is paid against; narrow ones fit
// the 13-, 14-, 27- and 28-column maps without ragged edges.
constexpr TileChoice kTiles5[] = {{4, 4, 7, 4}, {4, 3, 9, 4}, {4, 1, 28, 4}, {2, 2, 28, 4}, {2, 1, 28, 4},
                                  {1, 2, 28, 4}, {4, 1, 16, 4}, {2, 2, 16, 4}, {1, 2, 16, 4}, {4, 4, 7, 8}};
constexpr TileChoice kTiles3[] = {{6, 2, 13, 4}, {4, 2, 16, 4}, {6, 1, 16, 4}, {2, 2, 28, 4}, {2, 1, 28, 4},
                                  {4, 1, 28, 4}, {1, 2, 28, 4}, {1, 2, 16, 4}, {2, 4, 16, 4}, {2, 2, 28, 8}};
constexpr TileChoice kTiles1[] = {{6, 2, 13, 4}, {6, 1, 16, 4}, {4, 2, 16, 4}, {4, 1, 28, 4}, {2, 2, 28, 4},
                                  {1, 2, 16, 4}};

// Launchers of the kernels of one filter size (sparse_fring_r{1,3,5}.hip).
hipError_t launch_r1(const FringArgs &a, const TileChoice &tc, hipStream_t s);
hipError_t launch_r3(const FringArgs &a, const TileChoice &tc, hipStream_t s);
hipError_t launch_r5(const FringArgs &a, const TileChoice &tc, hipStream_t s);

}  // namespace fring
}  // namespace isc

#ifdef ISC_FRING_INSTANTIATE
namespace isc {
namespace fring {
namespace {

template <int RS_, int KPL, int TH, int TW, int NW>
struct FringShape {
    using T = tile::Shape<RS_, RS_, KPL, TH, TW>;
    static constexpr int kWaves = NW;
    static constexpr int RS2 = RS_ * RS_;
    static constexpr int CHF = RS2 * T::KW;                  // floats of one channel's weights
    static constexpr int NDW = (CHF + 255) / 256;            // 1 KB direct-to-LDS blocks
    static constexpr int SLOT4 = NDW * kLanes;               // float4 per ring slot
    static constexpr size_t SLOTB = sizeof(float4) * SLOT4;  // bytes of one stage's weights
    static constexpr int WIN4 = NW * T::EPL * kLanes / 4;    // float4 of its windows
    static constexpr size_t WINB = sizeof(float4) * WIN4;
    static constexpr int DPW = (NDW + NW - 1) / NW;          // weight blocks per wavefront per stage
    static constexpr int VPS = DPW + T::EPL;                 // vector-memory operations per stage
    // stages: up to 4 for slots of <= 16 KB, 3 for <= 32 KB, else 2, within
    // the workgroup's share of LDS (half of it for four wavefronts, so that
    // two workgroups share a CU) and few enough that the wait for the stage
    // consumed fits the vmcnt field.  Deeper rings measured slower: the LDS
    // they take costs resident workgroups (six stages for the inception 3x3
    // branch on 1 x 28 tiles: 0.205 -> 0.284 ms)
    static constexpr size_t BUDGET = NW == 4 ? kLdsMax / 2 : kLdsMax;
    static constexpr int NPREF = SLOTB <= 16384 ? 4 : (SLOTB <= 32768 ? 3 : 2);
    static constexpr int NFIT = static_cast<int>(BUDGET / (SLOTB + WINB));
    static constexpr int NVM = 63 / VPS + 2;
    static constexpr int NCAP = NFIT < NVM ? NFIT : NVM;
    static constexpr int NBUF = NPREF < NCAP ? NPREF : NCAP;
    static_assert(NBUF >= 2, "ring needs two stages");
    static constexpr size_t lds = NBUF * (SLOTB + WINB);
};

template <int RS_, int KPL, int TH, int TW, int NW>
__global__ __launch_bounds__(NW * kLanes)
void sparse_conv_fring_kernel(FringArgs a) {
    using SH = FringShape<RS_, KPL, TH, TW, NW>;
    constexpr int kWaves = NW;
    using T = typename SH::T;
    constexpr int KW = T::KW, NDW = SH::NDW, NBUF = SH::NBUF, DPW = SH::DPW, EPL = T::EPL;

    // ring of NBUF slots, each one channel's weights [R*S][KW] (k = kbase +
    // lane*KPL + j) padded to whole 1 KB blocks, then the wavefronts' input
    // windows [wavefront][q][lane].  Static, so that the compiler can tell
    // the slot being read from the slots being filled, and the kernel's only
    // LDS variable: with a second one the compiler makes every read of the
    // ring wait for all loads into LDS in flight, prefetched stages included.
    __shared__ float4 wring[NBUF][SH::SLOT4 + SH::WIN4];

    const int lane = threadIdx.x & (kLanes - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kLanes);
    const int kg = blockIdx.x % a.kgroups;
    // this wavefront's tile (past the last tile: the last tile's addresses,
    // nothing counted, nothing stored)
    const int tile = (blockIdx.x / a.kgroups) * kWaves + wave;
    const bool rows_ok = tile < a.ntiles;
    int t = rows_ok ? tile : a.ntiles - 1;
    const int ct = t % a.ctiles;
    t /= a.ctiles;
    const int band = t % a.rtiles;
    const int n = t / a.rtiles;
    const int oy0 = band * TH;
    const int ox0 = ct * TW;
    const int kbase = kg * KW;
    const int C = a.C, H = a.H, W = a.W, P = a.P, Kp = a.Kp;
    const int tw = min(TW, a.Wo - ox0);
    const size_t HW = static_cast<size_t>(H) * W;
    const float *x_n = a.x + static_cast<size_t>(n) * C * HW;

    // lane l of register q holds window element e = q*64 + l in leaf-key
    // order, e = wy * WCOLS + xp: input row oy0 - P + wy, column ox0 - P + xp.
    // Elements outside the map (padding) or past the window read the plane's
    // first element and never count as nonzero.
    int xoff[EPL];
    bool inwin[EPL];
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
        const int e = q * kLanes + lane;
        const int wy = e / T::WCOLS;
        const int y = oy0 - P + wy, xx = ox0 - P + (e - wy * T::WCOLS);
        inwin[q] = rows_ok && e < T::WROWS * T::WCOLS && y >= 0 && y < H && xx >= 0 && xx < W;
        xoff[q] = inwin[q] ? y * W + xx : 0;
    }

    // stage c -> slot SLOT: weights by direct global->LDS loads (every
    // wavefront issues exactly DPW blocks and EPL window loads, so the number
    // of vector-memory operations per stage is the same everywhere)
    auto issue = [&](auto slot_c, int c) {
        constexpr int SLOT = decltype(slot_c)::value;
#pragma unroll
        for (int i = 0; i < DPW; ++i) {
            const int d = min(wave + i * kWaves, NDW - 1);
            const int f = d * 256 + lane * 4;  // float offset in the slot
            int tap = f / KW;
            const int koff = f - tap * KW;
            tap = min(tap, SH::RS2 - 1);       // padding of the last block
            const int k = min(kbase + koff, Kp - 4);
            const float *src = a.wt + (static_cast<size_t>(c) * SH::RS2 + tap) * Kp + k;
            tile::load_lds16(src, &wring[SLOT][d * kLanes]);
        }
        const float *plane = x_n + static_cast<size_t>(c) * HW;
#pragma unroll
        for (int q = 0; q < EPL; ++q)
            tile::load_lds4(plane + xoff[q], reinterpret_cast<float *>(&wring[SLOT][SH::SLOT4]) + (wave * EPL + q) * kLanes);
    };

    // prologue: stages 0 .. NBUF-2 in flight before the decision is read
    // (past the last channel the last channel is loaded again, keeping the
    // per-stage operation count fixed)
    tile::static_for<0, NBUF - 1>([&](auto sl) { issue(sl, min(decltype(sl)::value, C - 1)); });
    const bool run = decision_gate(a.dec, 1u);
    if (!run) {
        __builtin_amdgcn_s_waitcnt(0);  // no load into LDS may outlive the workgroup
        return;
    }

    tile::Acc<T> acc;
#pragma unroll
    for (int y = 0; y < TH; ++y)
#pragma unroll
        for (int x = 0; x < TW; ++x)
#pragma unroll
            for (int j = 0; j < KPL; ++j) acc[y][x][j] = 0.0f;

    // per channel: wait for its stage and the barrier, issue the stage NBUF-1
    // channels ahead, then read the channel's weights and window (LDS ->
    // registers) into one set of registers, so that the scan (most of the
    // code) is inlined once
    float cur[EPL];
    tile::Wts<T> w;
#pragma unroll 1
    for (int c = 0; c < C; ++c) {
        tile::static_for<0, NBUF>([&](auto sl) {
            constexpr int B = decltype(sl)::value;
            if (c % NBUF == B) {
                // stage c complete for every wavefront; everyone is done with
                // stage c - 1, whose slot is refilled next
                tile::wait_vm_and_barrier<(NBUF - 2) * SH::VPS>();
                issue(std::integral_constant<int, (B + NBUF - 1) % NBUF>{}, min(c + NBUF - 1, C - 1));
                tile::load_weights<T>(reinterpret_cast<const float *>(&wring[B][0]), lane, w);
                const float *win = reinterpret_cast<const float *>(&wring[B][SH::SLOT4]) + wave * EPL * kLanes + lane;
#pragma unroll
                for (int q = 0; q < EPL; ++q) cur[q] = win[q * kLanes];
                tile::wait_lgkm0();
            }
        });
        unsigned long long mask[EPL];
#pragma unroll
        for (int q = 0; q < EPL; ++q) mask[q] = __ballot(inwin[q] && (__float_as_uint(cur[q]) & 0x7fffffffu) != 0u);
        tile::walk_scan<T>(mask, cur, acc, w);
    }
    __builtin_amdgcn_s_waitcnt(0);  // no load into LDS may outlive the workgroup

    // step 3: each lane stores its accumulators to NCHW
    uint32_t cnt = 0;
    if (rows_ok) {
        const size_t plane_out = static_cast<size_t>(a.Ho) * a.Wo;
        float *yrow = a.y + static_cast<size_t>(n) * a.K * plane_out + static_cast<size_t>(oy0) * a.Wo + ox0;
        cnt = tile::store_tile<T>(acc, yrow, plane_out, a.Wo, kbase, lane, a.K, a.Ho - oy0, tw, a.epi.relu);
    }
    if (a.epi.census) {
        __syncthreads();  // every wavefront is done with the ring
        census_commit(a.epi, cnt, reinterpret_cast<uint32_t *>(&wring[0][0]));
    }
}

template <int RS_, int KPL, int TH, int TW, int NW>
hipError_t launch_fring_t(const FringArgs &a, hipStream_t s) {
    if constexpr (!fring_fits(RS_, KPL, TH, TW)) {
        return hipErrorInvalidValue;
    } else {
        using SH = FringShape<RS_, KPL, TH, TW, NW>;
        constexpr int kWaves = NW;
        static_assert(SH::lds <= kLdsMax, "weight ring exceeds LDS");
        const int64_t grid = static_cast<int64_t>((a.ntiles + kWaves - 1) / kWaves) * a.kgroups;
        if (a.epi.census && census_slots_for(grid) > a.epi.cap) return hipErrorInvalidValue;
        sparse_conv_fring_kernel<RS_, KPL, TH, TW, NW><<<static_cast<unsigned>(grid), kWaves * kLanes, 0, s>>>(a);
        return hipGetLastError();
    }
}

// The launcher of table entry I of TILES when it is the chosen tile, else
// the next entry's.
template <int RS_, const TileChoice *TILES, int I, int NT>
hipError_t launch_fring_table(const FringArgs &a, const TileChoice &tc, hipStream_t s) {
    if constexpr (I >= NT) {
        return hipErrorInvalidValue;
    } else {
        constexpr TileChoice t = TILES[I];
        if (tc.kpl == t.kpl && tc.th == t.th && tc.tw == t.tw && tc.nw == t.nw)
            return launch_fring_t<RS_, t.kpl, t.th, t.tw, t.nw>(a, s);
        return launch_fring_table<RS_, TILES, I + 1, NT>(a, tc, s);
    }
}

template <int RS_>
hipError_t launch_fring_rs(const FringArgs &a, const TileChoice &tc, hipStream_t s) {
    if constexpr (RS_ == 5) {
        return launch_fring_table<5, kTiles5, 0, sizeof(kTiles5) / sizeof(kTiles5[0])>(a, tc, s);
    } else if constexpr (RS_ == 3) {
        return launch_fring_table<3, kTiles3, 0, sizeof(kTiles3) / sizeof(kTiles3[0])>(a, tc, s);
    } else {
        return launch_fring_table<1, kTiles1, 0, sizeof(kTiles1) / sizeof(kTiles1[0])>(a, tc, s);
    }
}

}  // namespace
}  // namespace fring
}  // namespace isc
#endif
