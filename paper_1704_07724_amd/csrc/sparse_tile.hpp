// Register-tile machinery shared by the zero-skipping kernels (ISC steps 2
// and 3, Sec. "Sparse Convolution"): square R x S filters, stride 1 (the
// filter-resident kernel also at stride 2).
//
// A wavefront owns an output tile of TH rows x TW columns x 64*KPL output
// maps: lane l accumulates maps kbase + l*KPL + j (j < KPL) in registers
// acc[oy][ox][j].  Lanes run over output maps as the paper's SIMD lanes do
// (step 2 multiplies one nonzero input by a K-contiguous weight vector), so
// every nonzero input is a wave-uniform scalar.  With the current channel's
// weights w[r][s][j] in registers, a nonzero at window row wy and shifted
// column xp adds v * w[r][s][j] to acc[wy - r][xp - s][j] for every tap that
// lands in the tile.  The position is data-dependent, so a compile-time
// binary dispatch on (wy, xp) selects a straight-line block whose register
// indices are constants: the inner loop has no memory operations, only the
// block's fused multiply-adds and a few scalar compares.
#pragma once

#include "isc_internal.hpp"
#include "dispatch_gen.hpp"

#include <type_traits>

namespace isc {
namespace tile {

constexpr int kLanes = 64;

// T_: the convolution's stride (output row oy reads input rows oy*T + r).
template <int R_, int S_, int KPL_, int TH_, int TW_, int T_ = 1>
struct Shape {
    static constexpr int R = R_, S = S_, KPL = KPL_, TH = TH_, TW = TW_, T = T_;
    static constexpr int KW = kLanes * KPL;           // output maps per wavefront
    static constexpr int WROWS = (TH - 1) * T + R;    // input rows the tile sees
    static constexpr int WCOLS = (TW - 1) * T + S;    // shifted input columns it sees
    // list entries of the tile's window, staged kLanes per register
    static constexpr int EPL = (WROWS * WCOLS + kLanes - 1) / kLanes;
};

template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

template <typename SH>
using Acc = float[SH::TH][SH::TW][SH::KPL];
template <typename SH>
using Wts = float[SH::R][SH::S][SH::KPL];

// Straight-line block for a nonzero at window row WY, shifted column XP:
// tap (r, s) reaches output ((WY - r) / T, (XP - s) / T) when both divide.
template <typename SH, int WY, int XP>
__device__ __forceinline__ void leaf(Acc<SH> &acc, const Wts<SH> &w, float v) {
#pragma unroll
    for (int r = 0; r < SH::R; ++r) {
        const int dy = WY - r;
        if (dy < 0 || dy % SH::T != 0 || dy / SH::T >= SH::TH) continue;
        const int oy = dy / SH::T;
#pragma unroll
        for (int s = 0; s < SH::S; ++s) {
            const int dx = XP - s;
            if (dx < 0 || dx % SH::T != 0 || dx / SH::T >= SH::TW) continue;
            const int ox = dx / SH::T;
#pragma unroll
            for (int j = 0; j < SH::KPL; ++j) acc[oy][ox][j] = __builtin_fmaf(v, w[r][s][j], acc[oy][ox][j]);
        }
    }
}

// Binary dispatch of the leaf key q = wy * WCOLS + xp in [LO, HI).
template <typename SH, int LO, int HI>
__device__ __forceinline__ void dispatch(int q, Acc<SH> &acc, const Wts<SH> &w, float v) {
    if constexpr (HI - LO == 1) {
        leaf<SH, LO / SH::WCOLS, LO % SH::WCOLS>(acc, w, v);
    } else {
        constexpr int MID = (LO + HI) / 2;
        if (q < MID)
            dispatch<SH, LO, MID>(q, acc, w, v);
        else
            dispatch<SH, MID, HI>(q, acc, w, v);
    }
}

// One nonzero: the computed-jump dispatch (generated inline assembly) for
// single-row one-map-per-lane tiles, whose leaves are short and whose trees
// are deepest; the binary tree otherwise (measured faster for taller tiles,
// whose leaves are long: the jump lands on a cold fetch of a padded leaf).
// ISC_TREE_DISPATCH selects the tree everywhere (for measurements).
#ifdef ISC_TREE_DISPATCH
constexpr bool kJumpDispatch = false;
#else
constexpr bool kJumpDispatch = true;
#endif

template <typename SH>
__device__ __forceinline__ void dispatch_one(int key, int vbits, Acc<SH> &acc, const Wts<SH> &w) {
    if constexpr (kJumpDispatch && SH::KPL == 1 && SH::R == SH::S && SH::TH == 1 &&
                  AsmDispatch<SH::R, SH::TH, SH::TW>::kAvailable) {
        AsmDispatch<SH::R, SH::TH, SH::TW>::run(key, vbits, acc, w);
    } else {
        dispatch<SH, 0, SH::WROWS * SH::WCOLS>(key, acc, w, __int_as_float(vbits));
    }
}

// Walk the first len entries of a run staged in registers (entry
// q*kLanes + l in lane l of run[q]); every entry lies in the tile's window
// rows [ybase, ybase + WROWS).  The lanes first turn their entries into leaf
// keys (wy * WCOLS + x + xshift, or -1 for a column outside [xlo, xlo +
// xspan] when CHECK_X), so that per nonzero the scalar unit only walks the
// dispatch tree.  Callers inline this once per kernel: the tree is most of
// the kernel's code.
template <typename SH, bool CHECK_X>
__device__ __forceinline__ void walk(const NzEntry (&run)[SH::EPL], int len, int ybase, int xshift, int xlo,
                                     int xspan, Acc<SH> &acc, const Wts<SH> &w) {
#pragma unroll
    for (int q = 0; q < SH::EPL; ++q) {
        const int cnt = min(len - q * kLanes, kLanes);
        if (cnt <= 0) break;
        const int yx = static_cast<int>(run[q].yx);
        const int x = yx & 0xffff;
        int key = ((yx >> 16) - ybase) * SH::WCOLS + x + xshift;
        if (CHECK_X && static_cast<unsigned>(x - xlo) > static_cast<unsigned>(xspan)) key = -1;
        const int vbits = __float_as_int(run[q].v);
#pragma unroll 1
        for (int jj = 0; jj < cnt; ++jj) {
            const int k = __builtin_amdgcn_readlane(key, jj);
            const int vb = __builtin_amdgcn_readlane(vbits, jj);
            if (!CHECK_X || k >= 0) dispatch_one<SH>(k, vb, acc, w);
        }
    }
}

// Walk the nonzeros flagged in a 64-bit wavefront mask (bit l: lane l holds
// a nonzero whose leaf key is keyv and whose value bits are vbits), in lane
// order.  Per nonzero: find-first-set, clear, two lane reads, the tree.
template <typename SH>
__device__ __forceinline__ void walk_mask(unsigned long long mask, int keyv, int vbits, Acc<SH> &acc,
                                          const Wts<SH> &w) {
#pragma unroll 1
    while (mask) {
        const int j = __builtin_ctzll(mask);
        mask &= mask - 1;
        dispatch_one<SH>(__builtin_amdgcn_readlane(keyv, j), __builtin_amdgcn_readlane(vbits, j), acc, w);
    }
}

// Static scan of a window laid out in leaf-key order (element q of the
// window, q = wy * WCOLS + xp, is lane q % 64 of xv[q / 64]): the positions
// are visited in order, in groups of 16, then 4, then one, each group tested
// against the mask and skipped when empty; a set position runs its
// straight-line block.  The tests are wave-uniform scalar branches laid out
// so that an empty group falls through (no fetch redirect), and there is no
// dependent chain from one nonzero to the next.
// The ballots as 32-bit halves, each through an opaque move so that the
// scan's tests stay 32-bit (a 64-bit test of a group inside one half costs
// a compare and a register move more): a single position is one bit test,
// a group one AND whose result decides the branch.
template <int EPL>
__device__ __forceinline__ void split_mask(const unsigned long long (&mask)[EPL], uint32_t (&mh)[2 * EPL]) {
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
        asm("s_mov_b32 %0, %1" : "=s"(mh[2 * e]) : "s"(static_cast<uint32_t>(mask[e])));
        asm("s_mov_b32 %0, %1" : "=s"(mh[2 * e + 1]) : "s"(static_cast<uint32_t>(mask[e] >> 32)));
    }
}

// Whether any of the N positions from lane L of ballot E are set (N <= 16,
// L a multiple of N: the group lies inside one half).
template <int E, int L, int N>
__device__ __forceinline__ bool group_set(const uint32_t *mh) {
    static_assert(N <= 16 && (L % 32) + N <= 32, "group crosses the 32-bit halves");
    constexpr uint32_t g = (N == 32 ? ~0u : ((1u << N) - 1u)) << (L % 32);
    return (mh[2 * E + L / 32] & g) != 0u;
}

template <typename SH, int Q>
__device__ __forceinline__ void scan_one(const uint32_t (&mh)[2 * SH::EPL], const float (&xv)[SH::EPL],
                                         Acc<SH> &acc, const Wts<SH> &w) {
    constexpr int E = Q / kLanes, L = Q % kLanes;
    if (__builtin_expect((mh[2 * E + L / 32] & (1u << (L % 32))) != 0u, 0)) {
        const float v = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(xv[E]), L));
        leaf<SH, Q / SH::WCOLS, Q % SH::WCOLS>(acc, w, v);
    }
}

// Positions [Q0, Q0 + G) (G a power of two dividing 64, clipped to the
// window), then the next level down.
template <typename SH, int Q0, int G>
__device__ __forceinline__ void scan_group(const uint32_t (&mh)[2 * SH::EPL], const float (&xv)[SH::EPL],
                                           Acc<SH> &acc, const Wts<SH> &w) {
    constexpr int NQ = SH::WROWS * SH::WCOLS;
    if constexpr (Q0 < NQ) {
        if constexpr (G == 1) {
            scan_one<SH, Q0>(mh, xv, acc, w);
        } else {
            constexpr int E = Q0 / kLanes, L = Q0 % kLanes;
            constexpr int N = (NQ - Q0) < G ? (NQ - Q0) : G;
            if (__builtin_expect(group_set<E, L, N>(mh), 0)) {
                constexpr int G2 = G == 16 ? 4 : 1;
                static_for<0, G / G2>([&](auto ic) {
                    scan_group<SH, Q0 + decltype(ic)::value * G2, G2>(mh, xv, acc, w);
                });
            }
        }
    }
}

template <typename SH>
__device__ __forceinline__ void walk_scan(const unsigned long long (&mask)[SH::EPL], const float (&xv)[SH::EPL],
                                          Acc<SH> &acc, const Wts<SH> &w) {
    constexpr int NQ = SH::WROWS * SH::WCOLS;
    uint32_t mh[2 * SH::EPL];
    split_mask<SH::EPL>(mask, mh);
    static_for<0, (NQ + 15) / 16>([&](auto gc) { scan_group<SH, decltype(gc)::value * 16, 16>(mh, xv, acc, w); });
}

// The same static scan with the block of a set position supplied by the
// caller: blk(integral_constant<WY>, integral_constant<XP>, v) for a nonzero v
// at window row WY, shifted column XP (the weight-gradient kernel's leaves).
template <typename SH, int Q, typename Blk>
__device__ __forceinline__ void scan_one_f(const uint32_t (&mh)[2 * SH::EPL], const float (&xv)[SH::EPL], Blk &blk) {
    constexpr int E = Q / kLanes, L = Q % kLanes;
    if (__builtin_expect((mh[2 * E + L / 32] & (1u << (L % 32))) != 0u, 0)) {
        const float v = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(xv[E]), L));
        blk(std::integral_constant<int, Q / SH::WCOLS>{}, std::integral_constant<int, Q % SH::WCOLS>{}, v);
    }
}

template <typename SH, int Q0, int G, typename Blk>
__device__ __forceinline__ void scan_group_f(const uint32_t (&mh)[2 * SH::EPL], const float (&xv)[SH::EPL], Blk &blk) {
    constexpr int NQ = SH::WROWS * SH::WCOLS;
    if constexpr (Q0 < NQ) {
        if constexpr (G == 1) {
            scan_one_f<SH, Q0>(mh, xv, blk);
        } else {
            constexpr int E = Q0 / kLanes, L = Q0 % kLanes;
            constexpr int N = (NQ - Q0) < G ? (NQ - Q0) : G;
            if (__builtin_expect(group_set<E, L, N>(mh), 0)) {
                constexpr int G2 = G == 16 ? 4 : 1;
                static_for<0, G / G2>([&](auto ic) {
                    scan_group_f<SH, Q0 + decltype(ic)::value * G2, G2>(mh, xv, blk);
                });
            }
        }
    }
}

template <typename SH, typename Blk>
__device__ __forceinline__ void walk_scan_f(const unsigned long long (&mask)[SH::EPL], const float (&xv)[SH::EPL],
                                            Blk &blk) {
    constexpr int NQ = SH::WROWS * SH::WCOLS;
    uint32_t mh[2 * SH::EPL];
    split_mask<SH::EPL>(mask, mh);
    static_for<0, (NQ + 15) / 16>([&](auto gc) { scan_group_f<SH, decltype(gc)::value * 16, 16>(mh, xv, blk); });
}

// Load one channel's weights for this lane: w[r][s][j] = wc[(r*S+s)*ld + lane*KPL + j]
// (ld = KW for the ring's layout, padded for the transposed one).
template <typename SH>
__device__ __forceinline__ void load_weights(const float *wc, int lane, Wts<SH> &w, int ld = SH::KW) {
#pragma unroll
    for (int r = 0; r < SH::R; ++r)
#pragma unroll
        for (int s = 0; s < SH::S; ++s)
#pragma unroll
            for (int j = 0; j < SH::KPL; ++j) w[r][s][j] = wc[(r * SH::S + s) * ld + lane * SH::KPL + j];
}

// 16 bytes per lane from global memory straight into LDS at dst + 16 * lane
// (dst wave-uniform).  A device function: the builtin has no host form, and
// host-side instantiation of a lambda calling it would drop the kernel.
__device__ __forceinline__ void load_lds16(const float *src, float4 *dst) {
    __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
}

// 4 bytes per lane from global memory straight into LDS at dst + 4 * lane.
__device__ __forceinline__ void load_lds4(const float *src, float *dst) {
    __builtin_amdgcn_global_load_lds(src, dst, 4, 0, 0);
}

// s_waitcnt vmcnt(VM) with lgkmcnt(0) when LGKM0, expcnt untouched.
template <int VM, bool LGKM0>
__device__ __forceinline__ void wait_vm() {
    static_assert(VM >= 0 && VM < 64, "vmcnt field");
    constexpr int imm = (VM & 0xF) | ((VM >> 4) << 14) | ((LGKM0 ? 0x0 : 0xF) << 8) | (0x7 << 4);
    __builtin_amdgcn_s_waitcnt(imm);
}

// s_waitcnt lgkmcnt(0): LDS reads issued so far have landed (placed after a
// channel's weight loads so that the dispatch tree's leaves need no waits).
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt((0x3F & 0xF) | (0x3 << 14) | (0x7 << 4)); }

// wait_vm<VM, lgkmcnt 0>, then a workgroup barrier that the compiler may not
// move memory operations across.
template <int VM>
__device__ __forceinline__ void wait_vm_and_barrier() {
    wait_vm<VM, true>();
    asm volatile("s_barrier" ::: "memory");
}

// Store the tile rows/columns inside the output (rows < rows_ok, columns <
// cols_ok) and maps < K to NCHW, rectified when relu is set; yrow points at
// y[n][0][oy0][ox0].  Returns how many of the stored values are nonzero.
template <typename SH>
__device__ __forceinline__ uint32_t store_tile(const Acc<SH> &acc, float *yrow, size_t plane_out, int Wo, int kbase,
                                               int lane, int K, int rows_ok, int cols_ok, int relu = 0) {
    uint32_t cnt = 0;
#pragma unroll
    for (int j = 0; j < SH::KPL; ++j) {
        const int k = kbase + lane * SH::KPL + j;
        if (k >= K) continue;
        float *dst = yrow + static_cast<size_t>(k) * plane_out;
#pragma unroll
        for (int oy = 0; oy < SH::TH; ++oy) {
            if (oy >= rows_ok) break;
#pragma unroll
            for (int ox = 0; ox < SH::TW; ++ox)
                if (ox < cols_ok) {
                    const float v = epilogue_value(acc[oy][ox][j], relu);
                    cnt += nonzero_bit(v);
                    dst[oy * Wo + ox] = v;
                }
        }
    }
    return cnt;
}

}  // namespace tile
}  // namespace isc
