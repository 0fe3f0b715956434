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
// image and share the filter.  Channels flow through a ring of NBUF stages:
// each stage's R*S*64*KPL weights go global -> LDS by direct loads (no
// staging registers), each wavefront's nonzero run for that channel goes into
// a matching ring of registers, and stages are issued NBUF-1 channels ahead;
// one barrier per channel, after a wait for exactly the stage consumed.  The
// compute phase reads only LDS and registers whose loads have completed.  At the end each lane stores its
// accumulators to NCHW (step 3).  Summation order per output is fixed (list
// order within a channel, channels in order), so results are deterministic.
#include "isc_internal.hpp"

#include <algorithm>
#include <cstdlib>
#include <type_traits>

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

// 16 bytes per lane from global memory straight into LDS at dst + 16 * lane
// (dst wave-uniform).  Kept in a device function: the builtin has no host
// form, and host-side instantiation of a lambda calling it would drop the
// kernel.
__device__ __forceinline__ void load_lds16(const float *src, float4 *dst) {
    __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
}

template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

// s_waitcnt vmcnt(VM) lgkmcnt(0) (expcnt untouched), then a workgroup
// barrier that the compiler may not move memory operations across.
template <int VM>
__device__ __forceinline__ void wait_vm_and_barrier() {
    static_assert(VM >= 0 && VM < 64, "vmcnt field");
    constexpr int imm = (VM & 0xF) | ((VM >> 4) << 14) | (0x7 << 4);  // lgkmcnt = 0
    __builtin_amdgcn_s_waitcnt(imm);
    asm volatile("s_barrier" ::: "memory");
}

template <int RS_, int KPL>
struct RegShape {
    static constexpr int KW = kLanes * KPL;                 // output maps per wavefront
    static constexpr int WFLOATS = RS_ * RS_ * KW;          // one channel's weights
    static constexpr int NDW = (WFLOATS + 255) / 256;       // 1 KB direct-to-LDS blocks
    static constexpr int SLOT4 = NDW * kLanes;              // float4 per ring slot
    // ring depth: deeper when a channel's weights are small
    static constexpr int NBUF = SLOT4 * 16 <= 8192 ? 4 : (SLOT4 * 16 <= 16384 ? 3 : 2);
    static constexpr int DPW = (NDW + kWaves - 1) / kWaves;  // weight blocks per wavefront
    static constexpr int EPL = kRunMax / kLanes;             // run entries per lane
    static constexpr int VPS = DPW + EPL;                    // vector-memory ops per stage
    static constexpr size_t lds_static = sizeof(float4) * NBUF * SLOT4;
};

template <int RS_, int KPL, int TWM>
__global__ __launch_bounds__(kWaves * kLanes)
void sparse_conv_reg_kernel(RegArgs a) {
    using SH = RegShape<RS_, KPL>;
    constexpr int R = RS_, S = RS_;
    constexpr int XMAX = TWM + S - 1;  // shifted columns a tile can see
    constexpr int KW = SH::KW, NDW = SH::NDW, NBUF = SH::NBUF, DPW = SH::DPW, EPL = SH::EPL;
    constexpr int NOFF = R + 1;        // row offsets kept per channel

    // ring of NBUF slots, each one channel's weights [R*S][KW] (k = kbase +
    // lane*KPL + j) padded to whole 1 KB blocks; static, so that the compiler
    // can tell the slot being read from the slots being filled
    __shared__ float4 wring[NBUF][SH::SLOT4];
    extern __shared__ int32_t offs_all[];  // [waves][C][R+1] row offsets

    const bool run_ok = decision_says_run(a.dec);
    if (blockIdx.x == 0 && threadIdx.x == 0 && a.dec.record) a.dec.record->path_taken = run_ok ? 1u : 2u;
    if (!run_ok) return;

    const int lane = threadIdx.x & (kLanes - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kLanes);
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
    const int C = a.C, H = a.H, P = a.P, Kp = a.Kp;
    const bool row_ok = oy < a.Ho;
    // input rows oy + r - P for r in [0, R), clipped to the map
    const int ylo = max(0, oy - P);
    const int yhi = min(H - 1, oy - P + R - 1);
    const int nrows = row_ok ? max(0, yhi - ylo + 1) : 0;
    const int tw = min(a.TW, a.Wo - ox0);
    const int xlo = max(0, ox0 - P);
    const int xhi = min(a.W - 1, ox0 + tw - 1 - P + S - 1);
    const size_t HW = static_cast<size_t>(H) * a.W;
    const NzEntry *nz_n = a.nz + static_cast<size_t>(n) * C * HW;
    int32_t *offs = offs_all + wave * C * NOFF;

    // row offsets of this wavefront's input rows, every channel
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

    // this wavefront's nonzero run of a channel (its R input rows, at most
    // kRunMax entries: the kernel is used only when R * W <= kRunMax), one
    // register ring slot per weight slot; lanes past the run read later
    // slots or the list's 256-entry tail and are ignored
    NzEntry run[NBUF][EPL];

    // stage c -> slot SLOT: weights by direct global->LDS loads (every
    // wavefront issues exactly DPW blocks and EPL run loads, so the number of
    // vector-memory operations per stage is the same everywhere)
    auto issue = [&](auto slot_c, int c) {
        constexpr int SLOT = decltype(slot_c)::value;
#pragma unroll
        for (int i = 0; i < DPW; ++i) {
            const int d = min(wave + i * kWaves, NDW - 1);
            const int f = d * 256 + lane * 4;  // float offset in the slot
            int tap = f / KW;
            const int koff = f - tap * KW;
            tap = min(tap, R * S - 1);         // padding of the last block
            const int k = min(kbase + koff, Kp - 4);
            const float *src = a.wt + (static_cast<size_t>(c) * R * S + tap) * Kp + k;
            load_lds16(src, &wring[SLOT][d * kLanes]);
        }
        const int e0 = __builtin_amdgcn_readfirstlane(offs[c * NOFF]);
        const NzEntry *rsrc = nz_n + static_cast<size_t>(c) * HW + e0 + lane;
#pragma unroll
        for (int q = 0; q < EPL; ++q) run[SLOT][q] = rsrc[q * kLanes];
    };

    // channel c from slot SLOT: LDS weights and register runs only
    auto compute = [&](auto slot_c, int c) {
        constexpr int SLOT = decltype(slot_c)::value;
        const float *wl = reinterpret_cast<const float *>(&wring[SLOT][0]);
        const int *oc = offs + c * NOFF;
        const int e0 = __builtin_amdgcn_readfirstlane(oc[0]);
        const int e_all = __builtin_amdgcn_readfirstlane(oc[nrows]) - e0;
        if (e_all <= 0) return;
        // one copy of the dispatch code: filter rows run as a loop, the row's
        // weights reloaded into the same registers
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
                for (int j = 0; j < KPL; ++j) w[s][j] = wl[(r * S + s) * KW + lane * KPL + j];
#pragma unroll 1
            for (int q0 = lo & ~(kLanes - 1); q0 < hi; q0 += kLanes) {
                const int qi = q0 / kLanes;
                NzEntry mine = run[SLOT][0];
#pragma unroll
                for (int q = 1; q < EPL; ++q)
                    if (qi == q) mine = run[SLOT][q];
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
    };

    // prologue: stages 0 .. NBUF-2 in flight (past the last channel the last
    // channel is loaded again, keeping the per-stage operation count fixed)
    static_for<0, NBUF - 1>([&](auto sl) { issue(sl, min(decltype(sl)::value, C - 1)); });
    for (int c0 = 0; c0 < C; c0 += NBUF) {
        static_for<0, NBUF>([&](auto sl) {
            constexpr int B = decltype(sl)::value;
            const int c = c0 + B;
            if (c < C) {
                // stage c complete for every wavefront; everyone is done with
                // stage c - 1, whose slot is refilled next
                wait_vm_and_barrier<(NBUF - 2) * SH::VPS>();
                issue(std::integral_constant<int, (B + NBUF - 1) % NBUF>{}, min(c + NBUF - 1, C - 1));
                compute(sl, c);
            }
        });
    }
    __builtin_amdgcn_s_waitcnt(0);  // no load into LDS may outlive the workgroup

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
    const size_t dyn = sizeof(int32_t) * kWaves * a.C * (RS_ + 1);
    if (RegShape<RS_, KPL>::lds_static + dyn > 160 * 1024) return hipErrorInvalidValue;
    auto kern = sparse_conv_reg_kernel<RS_, KPL, TWM>;
    if (RegShape<RS_, KPL>::lds_static + dyn > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(dyn));
        if (e != hipSuccess) return e;
    }
    const size_t lds = dyn;
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
    // LDS: the weight ring (at most 2 x 25 KB for the shapes instantiated)
    // and the row offsets of every channel
    const size_t lds = 64 * 1024 + sizeof(int32_t) * kWaves * sh.C * (sh.R + 1);
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
