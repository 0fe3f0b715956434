// Filter-ring kernel (sparse_fring.hpp): the choice of tile and the launch.
#include "sparse_fring.hpp"

#include <algorithm>
#include <cstdlib>

namespace isc {
namespace fring {
namespace {

// The compiled tiles of a filter size.
void tiles_for(int R, const TileChoice **t, int *n) {
    if (R == 5) {
        *t = kTiles5;
        *n = sizeof(kTiles5) / sizeof(kTiles5[0]);
    } else if (R == 3) {
        *t = kTiles3;
        *n = sizeof(kTiles3) / sizeof(kTiles3[0]);
    } else {
        *t = kTiles1;
        *n = sizeof(kTiles1) / sizeof(kTiles1[0]);
    }
}

// Relative cost of a tile on a shape, with the input assumed 90 % zero (the
// regime the sparse path is for).  Per channel and wavefront: the
// multiply-adds (taps per nonzero times maps per lane), the bytes the CU's
// LDS moves (the wavefront's weight reads and its share of the stage's
// direct loads) at 128 bytes a clock, the scan's scalar work per window
// position and per nonzero, and a fixed part (wait, barrier, ballot);
// windows are counted inside the map only.  Summed over the launch's
// wavefronts and divided over the CUs, less 15 % for every wavefront a SIMD
// holds beyond two (more latency hidden), and rounded up to whole
// rounds of resident workgroups.  The weights are those that ranked the
// compiled tiles on AlexNet conv2-5 and the inception 3x3 branch as measured.
double tile_cost(const SparseShape &sh, const TileChoice &t) {
    const double density = 0.1;
    const int64_t kw = static_cast<int64_t>(kLanes) * t.kpl;
    const int64_t kgroups = (sh.K + kw - 1) / kw;
    const int64_t ntiles = static_cast<int64_t>(sh.N) * ((sh.Ho + t.th - 1) / t.th) * ((sh.Wo + t.tw - 1) / t.tw);
    const int64_t wgs = (ntiles + t.nw - 1) / t.nw * kgroups;
    const int wrows = t.th + sh.R - 1, wcols = t.tw + sh.S - 1;
    const double win_in = static_cast<double>(std::min(wrows, sh.H)) * std::min(wcols, sh.W);
    const double useful = static_cast<double>(std::min(t.th, sh.Ho)) * std::min(t.tw, sh.Wo);
    const double taps = std::min<double>(sh.R * sh.S, useful * sh.R * sh.S / win_in);
    const double nz = density * win_in;
    const double fma = nz * taps * t.kpl;
    const double scan = 0.55 * wrows * wcols + 10.0 * nz;
    const double wbytes = 4.0 * sh.R * sh.S * kw;
    const int epl = (wrows * wcols + kLanes - 1) / kLanes;
    const double slot = wbytes + 256.0 * t.nw * epl;
    const double lds = (wbytes + slot / t.nw) / 128.0;
    const double per = fma + lds + scan + 60.0;
    const int regs = t.th * t.tw * t.kpl + sh.R * sh.S * t.kpl + 30;
    const int wps = std::min(8, 512 / ((regs + 7) / 8 * 8));  // wavefronts per SIMD
    const int64_t per_cu =
        std::max<int64_t>(1, std::min<int64_t>(4 * wps / t.nw, static_cast<int64_t>(2 * kLdsMax / (2.0 * slot))));
    const double rounds = static_cast<double>(wgs) / (256.0 * per_cu);
    const double fill = rounds / std::ceil(rounds);
    return static_cast<double>(wgs) * t.nw * sh.C * per / (1.0 + 0.15 * std::max(0, wps - 2)) / fill;
}

// The cheapest compiled tile that fits the register budget, restricted to a
// caller's maps_per_lane / rows / cols when those name a compiled tile.
bool fring_choose(const SparseShape &sh, TileChoice *tc) {
    const TileChoice *tiles;
    int n;
    tiles_for(sh.R, &tiles, &n);
    for (int pass = 0; pass < 2; ++pass) {
        const bool forced = pass == 0;
        if (forced && sh.tu.maps_per_lane <= 0 && sh.tu.rows <= 0 && sh.tu.cols <= 0 && sh.tu.waves <= 0) continue;
        bool found = false;
        double best = 0.0;
        for (int i = 0; i < n; ++i) {
            const TileChoice &t = tiles[i];
            if (t.nw != 4 && !(forced && sh.tu.waves == t.nw)) continue;  // eight only when asked for
            if (forced && ((sh.tu.maps_per_lane > 0 && t.kpl != sh.tu.maps_per_lane) ||
                           (sh.tu.rows > 0 && t.th != sh.tu.rows) || (sh.tu.cols > 0 && t.tw != sh.tu.cols) ||
                           (sh.tu.waves > 0 && t.nw != sh.tu.waves)))
                continue;
            if (!fring_fits(sh.R, t.kpl, t.th, t.tw)) continue;
            const double c = tile_cost(sh, t);
            if (!found || c < best) {
                *tc = t;
                best = c;
                found = true;
            }
        }
        if (found) return true;
    }
    return false;
}

}  // namespace
}  // namespace fring

bool sparse_fring_applies(const SparseShape &sh) {
    if (sh.T != 1 || sh.R != sh.S || !(sh.R == 1 || sh.R == 3 || sh.R == 5)) return false;
    fring::TileChoice tc;
    return fring::fring_choose(sh, &tc);
}

int64_t sparse_fring_max_groups(const SparseShape &sh) {
    using namespace fring;
    const TileChoice *tiles;
    int n;
    tiles_for(sh.R, &tiles, &n);
    int64_t most = 0;
    for (int i = 0; i < n; ++i) {
        const TileChoice &t = tiles[i];
        const int64_t ntiles =
            static_cast<int64_t>(sh.N) * ((sh.Ho + t.th - 1) / t.th) * ((sh.Wo + t.tw - 1) / t.tw);
        most = std::max(most, (ntiles + t.nw - 1) / t.nw * ((sh.K + kLanes * t.kpl - 1) / (kLanes * t.kpl)));
    }
    return most;
}

bool sparse_fring_plan_info(const SparseShape &sh, isc_plan *out) {
    using namespace fring;
    TileChoice tc;
    if (!sparse_fring_applies(sh) || !fring_choose(sh, &tc)) return false;
    const int64_t ntiles = static_cast<int64_t>(sh.N) * ((sh.Ho + tc.th - 1) / tc.th) * ((sh.Wo + tc.tw - 1) / tc.tw);
    const int64_t groups = (ntiles + tc.nw - 1) / tc.nw * ((sh.K + kLanes * tc.kpl - 1) / (kLanes * tc.kpl));
    *out = isc_plan{ISC_KERNEL_FUSED_RING, tc.th, tc.tw, tc.kpl, 1, tc.nw, groups};
    return true;
}

hipError_t launch_sparse_fring(const SparseShape &sh, const float *x, const float *wt, float *y, const Decision &dec,
                               hipStream_t s, const Epilogue &epi) {
    using namespace fring;
    TileChoice tc;
    if (sh.T != 1 || sh.R != sh.S || !fring_choose(sh, &tc)) return hipErrorInvalidValue;
    FringArgs a{};
    a.x = x;
    a.wt = wt;
    a.y = y;
    a.N = sh.N; a.C = sh.C; a.H = sh.H; a.W = sh.W; a.K = sh.K;
    a.Kp = (sh.K + kLanes - 1) / kLanes * kLanes;
    a.P = sh.P; a.Ho = sh.Ho; a.Wo = sh.Wo;
    a.ctiles = (sh.Wo + tc.tw - 1) / tc.tw;
    a.rtiles = (sh.Ho + tc.th - 1) / tc.th;
    const int64_t ntiles = static_cast<int64_t>(sh.N) * a.rtiles * a.ctiles;
    if (ntiles >= (1ll << 31) - tc.nw) return hipErrorInvalidValue;
    a.ntiles = static_cast<int>(ntiles);
    a.kgroups = (sh.K + kLanes * tc.kpl - 1) / (kLanes * tc.kpl);
    a.dec = dec;
    a.epi = epi;
    switch (sh.R) {
    case 1: return launch_r1(a, tc, s);
    case 3: return launch_r3(a, tc, s);
    default: return launch_r5(a, tc, s);
    }
}

}  // namespace isc
