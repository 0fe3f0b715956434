// ISC steps 2 and 3 (Sec. "Sparse Convolution"), register-tile kernel with
// the filter streamed through LDS: stride 1, square 1x1, 3x3 and 5x5
// filters, any number of input maps.
//
// A wavefront owns one output row (TH = 1), up to TW columns and 64*KPL
// output maps in registers (the tile machinery is described in
// sparse_tile.hpp).  The four wavefronts of a workgroup own four consecutive
// output rows of one image and share the filter.  Channels flow through a
// ring of NBUF LDS slots: a channel's R*S*64*KPL weights go global -> LDS by
// direct loads (no staging registers), each wavefront's nonzero run of that
// channel (its R input rows: one contiguous piece of the plane's row-major
// list) goes into a matching ring of registers, and stages are issued NBUF-1
// channels ahead; one barrier per channel, after a wait for exactly the stage
// consumed.  For each channel a wavefront loads the channel's weights from
// LDS into registers once and walks its whole run: every nonzero goes to the
// straight-line block of its (filter row, column).  At the end each lane
// stores its accumulators to NCHW (step 3).  Summation order per output is
// fixed (channels in order, list order within a channel), so results are
// deterministic.
#include "sparse_tile.hpp"

#include <algorithm>
#include <cstdlib>

namespace isc {
namespace {

using tile::kLanes;
constexpr int kWaves = 4;
constexpr int kRegBudget = 168;  // VGPRs for a channel's weights plus the tile

struct RingArgs {
    const int32_t *row_ptr;
    const NzEntry *nz;
    const float *wt;  // [C][R][S][Kp], K contiguous
    float *y;
    int N, C, H, W, K, Kp, P, Ho, Wo;
    int TWr;      // output columns per tile in use (<= TW)
    int ctiles;   // column tiles per row
    int bands;    // groups of kWaves output rows
    int kgroups;  // groups of 64 * KPL output maps
    Decision dec;
};

template <int RS_, int KPL, int TW>
struct RingShape {
    using T = tile::Shape<RS_, RS_, KPL, 1, TW>;
    static constexpr int CHF = RS_ * RS_ * T::KW;           // floats of one channel
    static constexpr int NDW = (CHF + 255) / 256;           // 1 KB direct-to-LDS blocks
    static constexpr int SLOT4 = NDW * kLanes;              // float4 per ring slot
    // ring depth: deeper when a channel's weights are small
    static constexpr int NBUF = SLOT4 * 16 <= 8192 ? 4 : (SLOT4 * 16 <= 16384 ? 3 : 2);
    static constexpr int DPW = (NDW + kWaves - 1) / kWaves;  // weight blocks per wavefront
    static constexpr int VPS = DPW + T::EPL;                 // vector-memory ops per stage
    static constexpr size_t lds_static = sizeof(float4) * NBUF * SLOT4;
};

template <int RS_, int KPL, int TW>
__global__ __launch_bounds__(kWaves * kLanes)
void sparse_conv_ring_kernel(RingArgs a) {
    using SH = RingShape<RS_, KPL, TW>;
    using T = typename SH::T;
    constexpr int R = RS_, S = RS_;
    constexpr int KW = T::KW, NDW = SH::NDW, NBUF = SH::NBUF, DPW = SH::DPW, EPL = T::EPL;
    constexpr int NOFF = R + 1;  // row offsets kept per channel

    // ring of NBUF slots, each one channel's weights [R*S][KW] (k = kbase +
    // lane*KPL + j) padded to whole 1 KB blocks; static, so that the compiler
    // can tell the slot being read from the slots being filled
    __shared__ float4 wring[NBUF][SH::SLOT4];
    extern __shared__ int32_t offs_all[];  // [waves][C][R+1] row offsets

    if (!decision_gate(a.dec, 1u)) return;

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
    const int ox0 = ct * a.TWr;
    const int kbase = kg * KW;
    const int C = a.C, H = a.H, P = a.P, Kp = a.Kp;
    const bool row_ok = oy < a.Ho;
    // input rows oy + r - P for r in [0, R), clipped to the map
    const int ylo = max(0, oy - P);
    const int yhi = min(H - 1, oy - P + R - 1);
    const int nrows = row_ok ? max(0, yhi - ylo + 1) : 0;
    const int tw = min(a.TWr, a.Wo - ox0);
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

    tile::Acc<T> acc;
#pragma unroll
    for (int x = 0; x < TW; ++x)
#pragma unroll
        for (int j = 0; j < KPL; ++j) acc[0][x][j] = 0.0f;

    // this wavefront's nonzero run of a channel, one register ring slot per
    // weight slot.  Lanes past the run re-read its last entry (no extra
    // lines); an empty run reads the slot it would start at, which the
    // list's 256-entry tail keeps in bounds.
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
            tile::load_lds16(src, &wring[SLOT][d * kLanes]);
        }
        const int e0 = __builtin_amdgcn_readfirstlane(offs[c * NOFF]);
        const int last = max(__builtin_amdgcn_readfirstlane(offs[c * NOFF + nrows]) - e0 - 1, 0);
        const NzEntry *rsrc = nz_n + static_cast<size_t>(c) * HW + e0;
#pragma unroll
        for (int q = 0; q < EPL; ++q) run[SLOT][q] = rsrc[min(q * kLanes + lane, last)];
    };

    // prologue: stages 0 .. NBUF-2 in flight (past the last channel the last
    // channel is loaded again, keeping the per-stage operation count fixed)
    tile::static_for<0, NBUF - 1>([&](auto sl) { issue(sl, min(decltype(sl)::value, C - 1)); });
    // per channel: wait for its stage and the barrier, issue the stage NBUF-1
    // channels ahead, then load the channel's weights (LDS -> registers) and
    // its run into one set of registers, so that the walk (most of the code)
    // is inlined once
    NzEntry cur[EPL];
    tile::Wts<T> w;
#pragma unroll 1
    for (int c = 0; c < C; ++c) {
        const int e0 = __builtin_amdgcn_readfirstlane(offs[c * NOFF]);
        const int len = __builtin_amdgcn_readfirstlane(offs[c * NOFF + nrows]) - e0;
        tile::static_for<0, NBUF>([&](auto sl) {
            constexpr int B = decltype(sl)::value;
            if (c % NBUF == B) {
                // stage c complete for every wavefront; everyone is done with
                // stage c - 1, whose slot is refilled next
                tile::wait_vm_and_barrier<(NBUF - 2) * SH::VPS>();
                issue(std::integral_constant<int, (B + NBUF - 1) % NBUF>{}, min(c + NBUF - 1, C - 1));
                if (len > 0) {
                    tile::load_weights<T>(reinterpret_cast<const float *>(&wring[B][0]), lane, w);
                    tile::wait_lgkm0();
#pragma unroll
                    for (int q = 0; q < EPL; ++q) cur[q] = run[B][q];
                }
            }
        });
        if (len > 0) tile::walk<T, true>(cur, len, oy - P, P - ox0, xlo, xhi - xlo, acc, w);
    }
    __builtin_amdgcn_s_waitcnt(0);  // no load into LDS may outlive the workgroup

    // step 3: each lane stores its accumulators to NCHW
    if (row_ok) {
        const size_t plane_out = static_cast<size_t>(a.Ho) * a.Wo;
        float *yrow = a.y + static_cast<size_t>(n) * a.K * plane_out + static_cast<size_t>(oy) * a.Wo + ox0;
        tile::store_tile<T>(acc, yrow, plane_out, a.Wo, kbase, lane, a.K, 1, tw);
    }
}

constexpr bool ring_fits(int RS, int KPL, int TW) { return (RS * RS + TW) * KPL <= kRegBudget; }

// Largest output maps per lane (1, 2, 4, 6) that K can use and that keeps a
// channel's weights and the tile within the register budget.
int ring_kpl(int K, int RS, int TW) {
    const int want = std::max((K + kLanes - 1) / kLanes, 1);
    for (int kpl : {6, 4, 2, 1})
        if (kpl <= want && ring_fits(RS, kpl, TW)) return kpl;
    return 1;
}

int ring_tw(int Wo) { return Wo <= 8 ? 8 : (Wo <= 16 ? 16 : 28); }

// List entries a wavefront stages: R rows of up to TW + R - 1 columns.
int ring_epl(int RS, int TW) { return (RS * (TW + RS - 1) + kLanes - 1) / kLanes; }

template <int RS_, int KPL, int TW>
hipError_t launch_ring_t(const RingArgs &a, hipStream_t s) {
    if constexpr (!ring_fits(RS_, KPL, TW)) {
        return hipErrorInvalidValue;
    } else {
        using SH = RingShape<RS_, KPL, TW>;
        const size_t dyn = sizeof(int32_t) * kWaves * a.C * (RS_ + 1);
        if (SH::lds_static + dyn > 160 * 1024) return hipErrorInvalidValue;
        auto kern = sparse_conv_ring_kernel<RS_, KPL, TW>;
        if (SH::lds_static + dyn > 64 * 1024) {
            hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(dyn));
            if (e != hipSuccess) return e;
        }
        const int grid = a.N * a.bands * a.ctiles * a.kgroups;
        kern<<<grid, kWaves * kLanes, dyn, s>>>(a);
        return hipGetLastError();
    }
}

template <int RS_, int TW>
hipError_t launch_ring_kpl(const RingArgs &a, int kpl, hipStream_t s) {
    switch (kpl) {
    case 1: return launch_ring_t<RS_, 1, TW>(a, s);
    case 2: return launch_ring_t<RS_, 2, TW>(a, s);
    case 4: return launch_ring_t<RS_, 4, TW>(a, s);
    default: return launch_ring_t<RS_, 6, TW>(a, s);
    }
}

template <int RS_>
hipError_t launch_ring_rs(const RingArgs &a, int kpl, int tw, hipStream_t s) {
    switch (tw) {
    case 8: return launch_ring_kpl<RS_, 8>(a, kpl, s);
    case 16: return launch_ring_kpl<RS_, 16>(a, kpl, s);
    default: return launch_ring_kpl<RS_, 28>(a, kpl, s);
    }
}

}  // namespace

bool sparse_ring_applies(const SparseShape &sh) {
    if (sh.T != 1 || sh.R != sh.S || !(sh.R == 1 || sh.R == 3 || sh.R == 5)) return false;
    // a wavefront's run (R whole input rows) must fit its staging registers
    const int tw = ring_tw(sh.Wo);
    if (static_cast<int64_t>(sh.R) * sh.W > static_cast<int64_t>(ring_epl(sh.R, tw)) * kLanes) return false;
    // LDS: the weight ring (at most 64 KB for the shapes instantiated) and
    // the row offsets of every channel
    const size_t lds = 64 * 1024 + sizeof(int32_t) * kWaves * sh.C * (sh.R + 1);
    return lds <= 160 * 1024;
}

hipError_t launch_sparse_ring(const SparseShape &sh, const int32_t *row_ptr, const NzEntry *nz, const float *wt,
                              float *y, const Decision &dec, hipStream_t s) {
    RingArgs a{};
    a.row_ptr = row_ptr;
    a.nz = nz;
    a.wt = wt;
    a.y = y;
    a.N = sh.N; a.C = sh.C; a.H = sh.H; a.W = sh.W; a.K = sh.K;
    a.Kp = (sh.K + kLanes - 1) / kLanes * kLanes;
    a.P = sh.P; a.Ho = sh.Ho; a.Wo = sh.Wo;
    const int tw = ring_tw(sh.Wo);
    int kpl = ring_kpl(sh.K, sh.R, tw);
    {  // a caller's override
        const int v = sh.tu.maps_per_lane;
        if ((v == 1 || v == 2 || v == 4 || v == 6) && ring_fits(sh.R, v, tw)) kpl = v;
    }
    a.TWr = std::min(tw, sh.Wo);
    a.ctiles = (sh.Wo + a.TWr - 1) / a.TWr;
    a.bands = (sh.Ho + kWaves - 1) / kWaves;
    a.kgroups = (sh.K + kLanes * kpl - 1) / (kLanes * kpl);
    a.dec = dec;
    switch (sh.R) {
    case 1: return launch_ring_rs<1>(a, kpl, tw, s);
    case 3: return launch_ring_rs<3>(a, kpl, tw, s);
    default: return launch_ring_rs<5>(a, kpl, tw, s);
    }
}

}  // namespace isc
