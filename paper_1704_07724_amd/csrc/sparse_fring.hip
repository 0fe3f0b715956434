// Filter-ring kernel (sparse_fring.hpp): the choice of tile and the launch.
#include "sparse_fring.hpp"

#include <algorithm>
#include <cstdlib>

namespace isc {
namespace fring {
namespace {

// Tiles of 16 or 28 columns (narrower maps use the 16-column tile), one or
// two rows per wavefront: the shapes the choice below takes in practice.
int fring_tw(int Wo) { return Wo <= 16 ? 16 : 28; }

// Among the tiles that fit the register budget, the one that wastes least
// work -- lanes past K in the last map group times rows past Ho in the last
// band.  Ties go to 4 maps per lane (256 maps per workgroup), then to two
// rows per wavefront (each weight read from LDS serves twice the outputs,
// which counts at high sparsity, where a channel's weight reads cost more
// than the few multiply-adds they feed), then to more maps per lane.  Tie
// order measured on AlexNet conv2-5 and the inception 3x3 branch; a caller's
// tuning maps_per_lane / rows restrict the choice.
bool fring_choose_fixed(const SparseShape &sh, int tw, int kpl_fix, int th_fix, TileChoice *tc) {
    bool found = false;
    double best = 0.0;
    int best_rank = 0;
    for (int kpl : {6, 4, 2, 1}) {
        if (kpl_fix > 0 && kpl != kpl_fix) continue;
        for (int th : {2, 1}) {
            if (th_fix > 0 && th != th_fix) continue;
            if (!fring_fits(sh.R, kpl, th, tw)) continue;
            const int kw = kLanes * kpl, rows = kWaves * th;
            const double lanes = static_cast<double>((sh.K + kw - 1) / kw * kw) / sh.K;
            const double rws = static_cast<double>((sh.Ho + rows - 1) / rows * rows) / sh.Ho;
            const double waste = lanes * rws;
            const int rank = (kpl == 4 ? 100 : 0) + th * 10 + kpl;  // tie order
            if (!found || waste < best * (1.0 - 1e-9) || (waste <= best * (1.0 + 1e-9) && rank > best_rank)) {
                *tc = TileChoice{kpl, th};
                best = waste;
                best_rank = rank;
                found = true;
            }
        }
    }
    return found;
}

// The caller's overrides when the shape takes them, else the choice above.
bool fring_choose(const SparseShape &sh, int tw, TileChoice *tc) {
    return fring_choose_fixed(sh, tw, sh.tu.maps_per_lane, sh.tu.rows, tc) || fring_choose_fixed(sh, tw, 0, 0, tc);
}

}  // namespace
}  // namespace fring

bool sparse_fring_applies(const SparseShape &sh) {
    if (sh.T != 1 || sh.R != sh.S || !(sh.R == 1 || sh.R == 3 || sh.R == 5)) return false;
    fring::TileChoice tc;
    return fring::fring_choose(sh, fring::fring_tw(sh.Wo), &tc);
}

bool sparse_fring_plan_info(const SparseShape &sh, isc_plan *out) {
    using namespace fring;
    const int tw = fring_tw(sh.Wo);
    TileChoice tc;
    if (!sparse_fring_applies(sh) || !fring_choose(sh, tw, &tc)) return false;
    const int twr = std::min(tw, sh.Wo);
    const int64_t groups = static_cast<int64_t>(sh.N) * ((sh.Ho + kWaves * tc.th - 1) / (kWaves * tc.th)) *
                           ((sh.Wo + twr - 1) / twr) * ((sh.K + kLanes * tc.kpl - 1) / (kLanes * tc.kpl));
    *out = isc_plan{ISC_KERNEL_FUSED_RING, tc.th, twr, tc.kpl, 1, kWaves, groups};
    return true;
}

hipError_t launch_sparse_fring(const SparseShape &sh, const float *x, const float *wt, float *y, const Decision &dec,
                               hipStream_t s, const Epilogue &epi) {
    using namespace fring;
    const int tw = fring_tw(sh.Wo);
    TileChoice tc;
    if (sh.T != 1 || sh.R != sh.S || !fring_choose(sh, tw, &tc)) return hipErrorInvalidValue;
    FringArgs a{};
    a.x = x;
    a.wt = wt;
    a.y = y;
    a.N = sh.N; a.C = sh.C; a.H = sh.H; a.W = sh.W; a.K = sh.K;
    a.Kp = (sh.K + kLanes - 1) / kLanes * kLanes;
    a.P = sh.P; a.Ho = sh.Ho; a.Wo = sh.Wo;
    a.TWr = std::min(tw, sh.Wo);
    a.ctiles = (sh.Wo + a.TWr - 1) / a.TWr;
    a.bands = (sh.Ho + kWaves * tc.th - 1) / (kWaves * tc.th);
    a.kgroups = (sh.K + kLanes * tc.kpl - 1) / (kLanes * tc.kpl);
    a.dec = dec;
    a.epi = epi;
    switch (sh.R) {
    case 1: return launch_r1(a, tw, tc, s);
    case 3: return launch_r3(a, tw, tc, s);
    default: return launch_r5(a, tw, tc, s);
    }
}

}  // namespace isc
