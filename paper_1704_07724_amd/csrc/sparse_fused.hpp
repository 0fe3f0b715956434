// Filter-resident kernel (declarations and, for the per-filter-size
// translation units that define ISC_FUSED_INSTANTIATE, the kernel and its
// launchers).
//
// ISC steps 1-3 (Sec. "Sparse Convolution") in one launch, for convolutions
// with square 1x1, 3x3 or 5x5 filters at stride 1 (3x3 and 5x5 also at
// stride 2 with at most 8 output columns) and at most 64 output maps (few
// input maps: LeNet conv2, an inception 5x5 branch, Tab. 2's LeNet conv2).
//
// The paper builds each input map's nonzero list on the fly before using it.
// Here the list never leaves the wavefront: a wavefront loads the input rows
// its output tile needs straight from x (coalesced, one element per lane),
// takes a 64-bit ballot of the zero test per 64 elements, and walks the set
// bits in lane order -- row-major order, the paper's list order -- reading
// each nonzero's value and leaf key from its lane.  There are no compacted
// lists or row offsets in memory.
//
// The filter comes in the K-contiguous layout of ISC step 2 (wt[crs][64],
// written by the repack); the workgroup copies all of it into LDS by direct
// global->LDS loads (no registers), and per channel a wavefront reads the
// channel's R*S weights (64 output maps, one per lane) into registers.
// Wavefront w owns a TH x TW output tile (tile machinery in sparse_tile.hpp)
// of row group w / cs and the input channels c = (w mod cs) + i*cs.  The cs
// partial tiles of a row group are then summed through LDS, phases p and
// p + cs/2 first, then those pairs in order, and stored to NCHW (step 3)
// with consecutive threads on consecutive columns of one output map.
// Summation order per output is fixed for a given launch shape, so results
// are deterministic.
#pragma once

#include "sparse_tile.hpp"

namespace isc {
namespace fused {

using tile::kLanes;
constexpr int kWaves = 8;
constexpr size_t kLdsMax = 160 * 1024;
constexpr int kRPad = 65;        // LDS pitch of one tile position's output maps (reduction)
static_assert(kRPad > kLanes, "the pad column holds the census sums");
constexpr int kMaxTile = 64;     // accumulators per lane
constexpr int kRegSlots = kWaves / 2;  // phase-pair tiles of the register-weight kernel's reduction
constexpr int kMinGroups = 256;  // workgroups that fill the CUs once
constexpr int kWPitch = 64;      // maps per filter column in the repacked layout (K <= 64)
// Word 3 of a raw buffer resource on gfx9-family chips (gfx950 included):
// 32-bit data format, no swizzle, bounds checked against the record count.
constexpr int kBufferFormat = 0x00020000;


struct FusedArgs {
    const float *x;   // N x C x H x W
    const float *wt;  // [C*R*S][64], output map fastest, zero past K
    float *y;         // N x K x Ho x Wo
    int N, C, H, W, K, P, Ho, Wo;
    int cs;           // channel phases per row group
    int rg;           // row groups per workgroup (kWaves / cs)
    int bands;        // groups of rg * TH output rows
    int kgroups;      // groups of 64 output maps (register-weight kernel; 1 otherwise)
    int Kp;           // maps per filter column of wt (K rounded up to 64)
    int wide;         // register-weight kernel: weights through a buffer resource
    Decision dec;
    Epilogue epi;     // rectifier and census of y
};

struct FusedPlan {
    int th, tw, cs;
    size_t lds;
    int st;       // stride (1, or 2 with 8-column tiles)
    bool wreg;    // weights streamed to registers (sparse_conv_fused_reg_kernel)
};

// Launchers of the kernels of one filter size (sparse_fused_r{1,3,5}.hip).
hipError_t launch_r1(const FusedArgs &a, const FusedPlan &p, hipStream_t s);
hipError_t launch_r3(const FusedArgs &a, const FusedPlan &p, hipStream_t s);
hipError_t launch_r5(const FusedArgs &a, const FusedPlan &p, hipStream_t s);

}  // namespace fused
}  // namespace isc

#ifdef ISC_FUSED_INSTANTIATE
namespace isc {
namespace fused {
namespace {

template <int RS_, int TH, int TW, int ST>
__global__ __launch_bounds__(kWaves * kLanes)
void sparse_conv_fused_kernel(FusedArgs a) {
    using T = tile::Shape<RS_, RS_, 1, TH, TW, ST>;
    constexpr int RS2 = RS_ * RS_, EPL = T::EPL;
    constexpr int NS = 4;  // input-window register ring

    // the filter [C*R*S][64] during the walk, then the phase tiles
    // [wave][TH*TW][kRPad]
    extern __shared__ float lds[];

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
    const size_t HW = static_cast<size_t>(H) * W;
    const float *x_n = a.x + static_cast<size_t>(n) * C * HW;
    // this wavefront's channels: phase, phase + cs, ...
    const int ncw = phase < C ? (C - 1 - phase) / cs + 1 : 0;

    // lane l of register q holds window element e = q*64 + l in leaf-key
    // order, e = wy * WCOLS + xp: input row oy0*ST - P + wy, column xp - P.
    // Elements outside the map (padding) or past the window read the plane's
    // first element and never count as nonzero.
    int xoff[EPL];
    bool inwin[EPL];
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
        const int e = q * kLanes + lane;
        const int wy = e / T::WCOLS;
        const int y = oy0 * ST - P + wy, xx = e - wy * T::WCOLS - P;
        inwin[q] = rows_ok && e < T::WROWS * T::WCOLS && y >= 0 && y < H && xx >= 0 && xx < W;
        xoff[q] = inwin[q] ? y * W + xx : 0;
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

    // the filter into LDS, in flight before the decision is read so that the
    // two latencies overlap: 1 KB blocks (4 filter columns) spread over the
    // wavefronts, then single 256-byte columns for a remainder
    {
        const int ncol = C * RS2;
        const int nblk = ncol >> 2;
        for (int b = wave; b < nblk; b += kWaves)
            tile::load_lds16(a.wt + b * 4 * kWPitch + lane * 4, reinterpret_cast<float4 *>(lds + b * 4 * kWPitch));
        for (int t = nblk * 4 + wave; t < ncol; t += kWaves)
            tile::load_lds4(a.wt + t * kWPitch + lane, lds + t * kWPitch);
    }

    const bool run = decision_gate(a.dec, 1u);
    // every wavefront's part of the filter has landed in LDS (also before an
    // early exit: no load into LDS may outlive the workgroup)
    tile::wait_vm<0, true>();
    if (!run) return;
    __syncthreads();

    tile::Acc<T> acc;
#pragma unroll
    for (int y = 0; y < TH; ++y)
#pragma unroll
        for (int x = 0; x < TW; ++x) acc[y][x][0] = 0.0f;

    // channels in order; the window NS-1 channels ahead is loaded before each
    // compute; the slot's values and the channel's weights are copied to one
    // set of registers so that the walk (most of the code) is inlined once
    float cur[EPL];
    tile::Wts<T> w;
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
        tile::load_weights<T>(lds + static_cast<size_t>(phase + i * cs) * RS2 * kWPitch, lane, w, kWPitch);
        tile::wait_lgkm0();
        tile::walk_scan<T>(mask, cur, acc, w);
    }

    // step 3: the cs phase tiles of each row group are summed through LDS
    // and stored to NCHW.  Every wavefront writes its tile [position][map]
    // with a padded pitch (conflict-free); then each thread takes one output
    // position of the workgroup and the maps k0, k0 + ostep, ..., so that
    // consecutive threads store consecutive positions of one map, and sums
    // the phases of each output in pairs.
    constexpr int TP = TH * TW;
    __syncthreads();  // every wavefront is done with its weights
    float *red = lds;
#pragma unroll
    for (int y = 0; y < TH; ++y)
#pragma unroll
        for (int x = 0; x < TW; ++x) red[(wave * TP + y * TW + x) * kRPad + lane] = acc[y][x][0];
    __syncthreads();
    const int Wo = a.Wo;
    const int oyb = band * a.rg * TH;             // first output row of the workgroup
    const int rows = min(a.rg * TH, a.Ho - oyb);  // its output rows
    const int npos = rows * Wo;                   // <= kWaves * kMaxTile = 512
    const int ostep = (kWaves * kLanes) / npos;
    const int k0 = tid / npos;
    const int pos = tid - k0 * npos;
    const int oyl = pos / Wo;
    const int ox = pos - oyl * Wo;
    const int g = oyl / TH;
    const size_t plane_out = static_cast<size_t>(a.Ho) * Wo;
    const float *src = red + ((g * cs) * TP + (oyl - g * TH) * TW + ox) * kRPad;
    float *dst = a.y + static_cast<size_t>(n) * a.K * plane_out + static_cast<size_t>(oyb) * Wo + pos;
    // phase p's partial at src + p * TP * kRPad.  Summed in pairs (p, p +
    // cs/2), pairs in order -- the order of the register-weight kernel's
    // reduction, so the two kernels agree bitwise where both apply.  Pairs
    // past cs/2 read the last phase again (in bounds, no branches) and are
    // not added.
    const int h = cs > 1 ? cs / 2 : 0;
    int pa[kRegSlots], pb[kRegSlots];
#pragma unroll
    for (int i = 0; i < kRegSlots; ++i) {
        pa[i] = min(i, cs - 1) * TP * kRPad;
        pb[i] = min(i + h, cs - 1) * TP * kRPad;
    }
    const int relu = a.epi.relu;
    uint32_t cnt = 0;
    // threads past ostep map groups have no output (k0 >= ostep)
    for (int k = k0 < ostep ? k0 : a.K; k < a.K; k += ostep) {
        float pair[kRegSlots];
#pragma unroll
        for (int i = 0; i < kRegSlots; ++i) pair[i] = h > 0 ? src[pa[i] + k] + src[pb[i] + k] : src[pa[i] + k];
        float sum = pair[0];
#pragma unroll
        for (int i = 1; i < kRegSlots; ++i) sum += i < h ? pair[i] : 0.0f;
        sum = epilogue_value(sum, relu);
        cnt += nonzero_bit(sum);
        dst[static_cast<size_t>(k) * plane_out] = sum;
    }
    if (a.epi.census) {
        // the wavefront sums in the pad word of the first phase-tile rows
        // (column 64, which no tile store or read touches): no wait for the
        // reads above
        census_commit(a.epi, cnt, reinterpret_cast<uint32_t *>(red + kLanes), kRPad);
    }
}

// Variant for plans whose wavefronts share no input channel (cs == kWaves:
// one row group, every wavefront its own channels): each wavefront streams
// its channels' weights from the repacked filter (through L2) into
// registers, one channel ahead of its walk, so LDS holds only the tiles of
// the reduction -- one per pair of phases, for four-row tiles of 8 columns
// little enough for four workgroups per CU.  One workgroup per group of
// 64 output maps (kgroups), lanes over the maps of its group.  Stride 1;
// otherwise as the kernel above.
template <int RS_, int TH, int TW, bool WIDE>
__global__ __launch_bounds__(kWaves * kLanes, 4)
void sparse_conv_fused_reg_kernel(FusedArgs a) {
    using T = tile::Shape<RS_, RS_, 1, TH, TW>;
    constexpr int RS2 = RS_ * RS_, EPL = T::EPL;
    extern __shared__ float lds[];  // the phase-pair tiles [kRegSlots][TH*TW][kRPad]

    const int tid = threadIdx.x;
    const int lane = tid & (kLanes - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kLanes);
    const int cs = kWaves;
    const int phase = wave;
    const int kg = blockIdx.x % a.kgroups;  // this workgroup's 64 output maps
    const int rest = blockIdx.x / a.kgroups;
    const int band = rest % a.bands;
    const int n = rest / a.bands;
    const int oy0 = band * TH;
    const int kbase = kg * kLanes;
    const int kcnt = min(kLanes, a.K - kbase);
    const int C = a.C, H = a.H, W = a.W, P = a.P;
    const bool rows_ok = oy0 < a.Ho;
    const size_t HW = static_cast<size_t>(H) * W;
    const float *x_n = a.x + static_cast<size_t>(n) * C * HW;
    const int ncw = phase < C ? (C - 1 - phase) / cs + 1 : 0;

    int xoff[EPL];
    bool inwin[EPL];
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
        const int e = q * kLanes + lane;
        const int wy = e / T::WCOLS;
        const int y = oy0 - P + wy, xx = e - wy * T::WCOLS - P;
        inwin[q] = rows_ok && e < T::WROWS * T::WCOLS && y >= 0 && y < H && xx >= 0 && xx < W;
        xoff[q] = inwin[q] ? y * W + xx : 0;
    }

    // the next channel's window and weights (loaded a channel ahead; the
    // last channel is loaded again past the end, keeping every load in
    // bounds).  One group of maps (WIDE false): the taps 64 floats apart,
    // immediate offsets of one address.  Several (WIDE true): through a
    // buffer resource over the repacked filter (its size checked below 2^31
    // bytes by the plan), where the byte offset of tap t, t * Kp * 4, is the
    // same for every channel and stays in a scalar register, and the
    // channel's offset is one vector add, so a channel's RS2 loads take no
    // address arithmetic of their own.
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(a.wt), 0, C * RS2 * a.Kp * static_cast<int>(sizeof(float)), kBufferFormat);
    const int kp4 = a.Kp * static_cast<int>(sizeof(float));
    float xn[EPL];
    float wn[RS2];
    auto load_ch = [&](int i) {
        const int c = phase + min(i, ncw - 1) * cs;
        const float *plane = x_n + static_cast<size_t>(c) * HW;
#pragma unroll
        for (int q = 0; q < EPL; ++q) xn[q] = plane[xoff[q]];
        if constexpr (WIDE) {
            const int voff = ((c * RS2 * a.Kp + kbase + lane) * static_cast<int>(sizeof(float)));
#pragma unroll
            for (int t = 0; t < RS2; ++t)
                wn[t] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(wres, voff, t * kp4, 0));
        } else {
            const float *wc = a.wt + static_cast<size_t>(c) * RS2 * kWPitch + lane;
#pragma unroll
            for (int t = 0; t < RS2; ++t) wn[t] = wc[t * kWPitch];
        }
    };
    if (ncw > 0) load_ch(0);

    const bool run = decision_gate(a.dec, 1u);
    if (!run) {
        __builtin_amdgcn_s_waitcnt(0);
        return;
    }

    tile::Acc<T> acc;
#pragma unroll
    for (int y = 0; y < TH; ++y)
#pragma unroll
        for (int x = 0; x < TW; ++x) acc[y][x][0] = 0.0f;

#pragma unroll 1
    for (int i = 0; i < ncw; ++i) {
        // this channel's registers by explicit moves (which the compiler
        // cannot forward, so the loaded registers are free for the next
        // channel's loads and need no copy at the back edge), then the next
        // channel's loads fly during this channel's walk
        float cur[EPL];
        tile::Wts<T> w;
#pragma unroll
        for (int q = 0; q < EPL; ++q) asm volatile("v_mov_b32 %0, %1" : "=v"(cur[q]) : "v"(xn[q]));
#pragma unroll
        for (int t = 0; t < RS2; ++t) asm volatile("v_mov_b32 %0, %1" : "=v"(w[t / RS_][t % RS_][0]) : "v"(wn[t]));
        if (i + 1 < ncw) load_ch(i + 1);
        unsigned long long mask[EPL];
#pragma unroll
        for (int q = 0; q < EPL; ++q) mask[q] = __ballot(inwin[q] && (__float_as_uint(cur[q]) & 0x7fffffffu) != 0u);
        tile::walk_scan<T>(mask, cur, acc, w);
    }

    // step 3: the phase tiles summed through LDS and stored to NCHW, as in
    // the kernel above (one row group).  Half as many tiles as phases: the
    // upper phases write theirs, each lower phase p adds phase p + 4's to its
    // registers and writes the pair back into the same slot, and the store
    // sums the four pairs in order -- a fixed order, so deterministic.  The
    // smaller LDS footprint lets twice as many workgroups share a CU.
    constexpr int TP = TH * TW;
    constexpr int kSlots = kRegSlots;
    float *red = lds;
    const int slot = wave % kSlots;
    if (wave >= kSlots) {
#pragma unroll
        for (int y = 0; y < TH; ++y)
#pragma unroll
            for (int x = 0; x < TW; ++x) red[(slot * TP + y * TW + x) * kRPad + lane] = acc[y][x][0];
    }
    __syncthreads();
    if (wave < kSlots) {
#pragma unroll
        for (int y = 0; y < TH; ++y)
#pragma unroll
            for (int x = 0; x < TW; ++x) {
                float *r = red + (slot * TP + y * TW + x) * kRPad + lane;
                *r = acc[y][x][0] + *r;
            }
    }
    __syncthreads();
    const int Wo = a.Wo;
    const int rows = min(TH, a.Ho - oy0);
    const int npos = rows * Wo;  // <= kMaxTile
    const int ostep = (kWaves * kLanes) / npos;
    const int k0 = tid / npos;
    const int pos = tid - k0 * npos;
    const int oyl = pos / Wo;
    const int ox = pos - oyl * Wo;
    const size_t plane_out = static_cast<size_t>(a.Ho) * Wo;
    const float *src = red + (oyl * TW + ox) * kRPad;
    float *dst = a.y + (static_cast<size_t>(n) * a.K + kbase) * plane_out + static_cast<size_t>(oy0) * Wo + pos;
    const int relu = a.epi.relu;
    uint32_t cnt = 0;
    // k: map within this workgroup's group of 64
    for (int k = k0 < ostep ? k0 : kcnt; k < kcnt; k += ostep) {
        float part[kSlots];
#pragma unroll
        for (int p = 0; p < kSlots; ++p) part[p] = src[p * TP * kRPad + k];
        float sum = part[0];
#pragma unroll
        for (int p = 1; p < kSlots; ++p) sum += part[p];
        sum = epilogue_value(sum, relu);
        cnt += nonzero_bit(sum);
        dst[static_cast<size_t>(k) * plane_out] = sum;
    }
    if (a.epi.census) census_commit(a.epi, cnt, reinterpret_cast<uint32_t *>(red + kLanes), kRPad);
}

template <int RS_, int TH, int TW, bool WIDE>
hipError_t launch_fused_reg_w(const FusedArgs &a, size_t lds, hipStream_t s) {
    auto kern = sparse_conv_fused_reg_kernel<RS_, TH, TW, WIDE>;
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (e != hipSuccess) return e;
    }
    const int64_t grid = static_cast<int64_t>(a.N) * a.bands * a.kgroups;
    if (a.epi.census && census_slots_for(grid) > a.epi.cap) return hipErrorInvalidValue;
    kern<<<static_cast<unsigned>(grid), kWaves * kLanes, lds, s>>>(a);
    return hipGetLastError();
}

// one group of 64 maps: filter taps at immediate offsets (kgroups == 1 and
// Kp == 64); else, or when the caller asks (a.wide), through the buffer
// resource.
template <int RS_, int TH, int TW>
hipError_t launch_fused_reg_t(const FusedArgs &a, size_t lds, hipStream_t s) {
    return a.wide ? launch_fused_reg_w<RS_, TH, TW, true>(a, lds, s) : launch_fused_reg_w<RS_, TH, TW, false>(a, lds, s);
}

template <int RS_, int TH, int TW, int ST>
hipError_t launch_fused_t(const FusedArgs &a, size_t lds, hipStream_t s) {
    if constexpr (TH * TW > kMaxTile) {
        return hipErrorInvalidValue;
    } else {
        auto kern = sparse_conv_fused_kernel<RS_, TH, TW, ST>;
        if (lds > 64 * 1024) {
            hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
            if (e != hipSuccess) return e;
        }
        const int64_t grid = static_cast<int64_t>(a.N) * a.bands;
        if (a.epi.census && census_slots_for(grid) > a.epi.cap) return hipErrorInvalidValue;
        kern<<<static_cast<unsigned>(grid), kWaves * kLanes, lds, s>>>(a);
        return hipGetLastError();
    }
}

template <int RS_, int TW, int ST>
hipError_t launch_fused_th(const FusedArgs &a, int th, size_t lds, hipStream_t s) {
    switch (th) {
    case 8: return launch_fused_t<RS_, 8, TW, ST>(a, lds, s);
    case 4: return launch_fused_t<RS_, 4, TW, ST>(a, lds, s);
    case 2: return launch_fused_t<RS_, 2, TW, ST>(a, lds, s);
    default: return launch_fused_t<RS_, 1, TW, ST>(a, lds, s);
    }
}

// Stride 1 with 8-, 16- or 28-column tiles; stride 2 with 8-column tiles
// (3x3 and 5x5 filters).
template <int RS_>
hipError_t launch_fused_rs(const FusedArgs &a, const FusedPlan &p, hipStream_t s) {
    if (p.wreg) {
        // 4 x 8, 2 x 8, 2 x 16, 1 x 16 and the exact 13- and 14-column
        // tiles, stride 1
        if (p.st != 1) return hipErrorInvalidValue;
        if (p.tw == 8) {
            return p.th == 4 ? launch_fused_reg_t<RS_, 4, 8>(a, p.lds, s)
                             : (p.th == 2 ? launch_fused_reg_t<RS_, 2, 8>(a, p.lds, s) : hipErrorInvalidValue);
        }
        if (p.tw == 16) {
            return p.th == 2 ? launch_fused_reg_t<RS_, 2, 16>(a, p.lds, s)
                             : (p.th == 1 ? launch_fused_reg_t<RS_, 1, 16>(a, p.lds, s) : hipErrorInvalidValue);
        }
        if (p.tw == 13) {
            return p.th == 2 ? launch_fused_reg_t<RS_, 2, 13>(a, p.lds, s)
                             : (p.th == 1 ? launch_fused_reg_t<RS_, 1, 13>(a, p.lds, s) : hipErrorInvalidValue);
        }
        if (p.tw == 14) {
            return p.th == 2 ? launch_fused_reg_t<RS_, 2, 14>(a, p.lds, s)
                             : (p.th == 1 ? launch_fused_reg_t<RS_, 1, 14>(a, p.lds, s) : hipErrorInvalidValue);
        }
        return hipErrorInvalidValue;
    }
    if (p.st == 2) {
        if constexpr (RS_ == 1) {
            return hipErrorInvalidValue;
        } else {
            return p.tw == 8 ? launch_fused_th<RS_, 8, 2>(a, p.th, p.lds, s) : hipErrorInvalidValue;
        }
    }
    switch (p.tw) {
    case 8: return launch_fused_th<RS_, 8, 1>(a, p.th, p.lds, s);
    case 16: return launch_fused_th<RS_, 16, 1>(a, p.th, p.lds, s);
    default: return launch_fused_th<RS_, 28, 1>(a, p.th, p.lds, s);
    }
}

}  // namespace
}  // namespace fused
}  // namespace isc
#endif
