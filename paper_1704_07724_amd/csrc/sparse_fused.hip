// Filter-resident kernel (sparse_fused.hpp): the plan, the launch, and the
// choice between it and the filter-ring kernel.
#include "sparse_fused.hpp"

#include <algorithm>
#include <cstdlib>

namespace isc {
namespace fused {
namespace {

int fused_tw(int Wo) { return Wo <= 8 ? 8 : (Wo <= 16 ? 16 : 28); }

size_t fused_lds(int crs, int th, int tw) {
    return std::max(sizeof(float) * crs * kWPitch, sizeof(float) * kWaves * th * tw * kRPad);
}

// Plans whose wavefronts share no channel (every wavefront its own phase)
// gain nothing from the filter in LDS: with the weights streamed to
// registers, LDS holds only the reduction's tiles, and 32-position tiles let
// two workgroups share a CU (LeNet conv2: 13.2 -> 9.5 us), four since the
// tiles are summed in pairs (AlexNet conv3-5 10-12 % faster).  The filter need not
// fit in LDS at all, and one workgroup per group of 64 maps takes any K
// (AlexNet-ImageNet conv4 of Tab. 2 at batch 128: 259 us on the
// filter-ring kernel -> 113 us).  Taken wherever eligible: stride 1, square
// 1x1, 3x3 and 5x5 filters, at most 16 output columns.  A caller's tuning
// kernel FUSED or FUSED_RING keeps the filter in LDS, or in the ring beyond
// 64 maps.
bool fused_wreg_plan(const SparseShape &sh, FusedPlan *plan) {
    if (sh.tu.kernel == ISC_KERNEL_FUSED || sh.tu.kernel == ISC_KERNEL_FUSED_RING) return false;
    if (sh.T != 1 || sh.Wo > 16) return false;
    // the kernel addresses the repacked filter with 32-bit byte offsets
    const int64_t kp = (sh.K + kLanes - 1) / kLanes * kLanes;
    if (static_cast<int64_t>(sh.C) * sh.R * sh.S * kp * static_cast<int64_t>(sizeof(float)) >= (1ll << 31))
        return false;
    // 4 x 8 or 2 x 16 tiles, 2 x 13 and 2 x 14 on maps of exactly that width
    // (AlexNet conv3-5, the 14 x 14 inception layers: the window loses the
    // columns past the map and fits one ballot; conv3-5 5 % faster); half as
    // many rows when full ones leave CUs without a workgroup (LeNet conv2 at
    // batch 8: 7.7 -> 6.4 us; at batch 256 they cost 44 %).  A caller's
    // tuning rows fixes the rows.
    const int tw = sh.Wo <= 8 ? 8 : (sh.Wo == 13 || sh.Wo == 14 ? sh.Wo : 16);
    const int full = 32 / tw;
    const int64_t kgroups = (sh.K + kLanes - 1) / kLanes;
    int th = static_cast<int64_t>(sh.N) * ((sh.Ho + full - 1) / full) * kgroups < kMinGroups ? full / 2 : full;
    if (sh.tu.rows == full || sh.tu.rows == full / 2) th = sh.tu.rows;
    *plan = FusedPlan{th, tw, kWaves, sizeof(float) * kRegSlots * th * tw * kRPad, 1, true};
    return true;
}

// The filter must fit in LDS; stride 1, or stride 2 with 3x3 or 5x5 filters
// and at most 8 output columns.  Tile height and channel phases: the tallest
// tile (up to kMaxTile accumulators per lane), then the fewest phases that
// leave no row group of a workgroup idle (rg <= ceil(Ho / TH)), preferring
// plans with at least kMinGroups workgroups; else the plan with most
// workgroups.  A caller's tuning rows caps the tile height and phases fixes
// the phases; tuning kernel FUSED_RING leaves the shape to the filter-ring
// kernel.
bool fused_plan(const SparseShape &sh, FusedPlan *plan) {
    if (sh.tu.kernel == ISC_KERNEL_FUSED_RING && sparse_fring_applies(sh)) return false;
    if (sh.R != sh.S || !(sh.R == 1 || sh.R == 3 || sh.R == 5)) return false;
    if (!(sh.T == 1 || (sh.T == 2 && sh.R > 1 && sh.Wo <= 8))) return false;
    if (sh.Wo > 28) return false;
    // beyond 64 maps only the register-weight kernel (one wavefront per 64
    // maps and channel phase), where it takes the shape and the caller does
    // not ask for the filter-ring kernel: at 13 x 13 and sparsity 0.95
    // (AlexNet conv3-5) it beat every tile of the filter-ring kernel by
    // 12-30 %, the ring's tiles of up to 384 maps leaving CUs idle or
    // waiting on each channel's stage
    if (sh.K > kLanes) return fused_wreg_plan(sh, plan);
    const int crs = sh.C * sh.R * sh.S;
    // a filter too large for LDS: only the register-weight kernel, which
    // keeps none of it there, takes it (one phase per wavefront)
    if (static_cast<size_t>(crs) * kWPitch * sizeof(float) > kLdsMax) return fused_wreg_plan(sh, plan);
    const int tw = fused_tw(sh.Wo);
    const int th_cap = sh.tu.rows > 0 ? sh.tu.rows : 8;
    const int cs_fix = sh.tu.phases == 1 || sh.tu.phases == 2 || sh.tu.phases == 4 || sh.tu.phases == 8 ? sh.tu.phases : 0;
    bool found = false, done = false;
    int64_t best_groups = 0;
    for (int th : {8, 4, 2, 1}) {
        if (th * tw > kMaxTile || th > th_cap) continue;
        const int rows_need = (sh.Ho + th - 1) / th;
        for (int cs : {1, 2, 4, 8}) {
            if (cs_fix > 0 && cs != cs_fix) continue;
            const int rg = kWaves / cs;
            if (cs_fix == 0 && rg > rows_need && cs < kWaves) continue;  // idle row groups
            const int64_t groups = static_cast<int64_t>(sh.N) * ((sh.Ho + rg * th - 1) / (rg * th));
            const size_t lds = fused_lds(crs, th, tw);
            if (lds > kLdsMax) continue;
            if (!found || groups > best_groups) {
                *plan = FusedPlan{th, tw, cs, lds, sh.T, false};
                best_groups = groups;
                found = true;
            }
            done = groups >= kMinGroups;
            break;  // more phases only add partial tiles
        }
        if (done) break;
    }
    if (found && plan->cs == kWaves) fused_wreg_plan(sh, plan);
    return found;
}

}  // namespace
}  // namespace fused

// The filter-resident kernel launches N * bands <= N * Ho workgroups; its
// register-weight variant N * bands * map groups, with bands <= Ho; the
// filter-ring kernel at most what its largest grid over its compiled tiles
// is (sparse_fring_max_groups).
int64_t sparse_fused_max_groups(const SparseShape &sh) {
    const int64_t reg = static_cast<int64_t>(sh.N) * sh.Ho * ((sh.K + 63) / 64);  // register-weight kernel
    return std::max(reg, sparse_fring_max_groups(sh));
}

bool sparse_fused_applies(const SparseShape &sh) {
    fused::FusedPlan p;
    return fused::fused_plan(sh, &p) || sparse_fring_applies(sh);
}

int sparse_fused_kernel(const SparseShape &sh) {
    fused::FusedPlan p;
    if (fused::fused_plan(sh, &p)) return p.wreg ? 6 : 1;
    return sparse_fring_applies(sh) ? 5 : 0;
}

bool sparse_fused_plan_info(const SparseShape &sh, isc_plan *out) {
    using namespace fused;
    FusedPlan p;
    if (!fused_plan(sh, &p)) return sparse_fring_plan_info(sh, out);
    const int rg = kWaves / p.cs;
    const int64_t bands = (sh.Ho + rg * p.th - 1) / (rg * p.th);
    const int64_t kgroups = p.wreg ? (sh.K + kLanes - 1) / kLanes : 1;
    *out = isc_plan{p.wreg ? ISC_KERNEL_FUSED_REG : ISC_KERNEL_FUSED, p.th, p.tw, 1, p.cs, kWaves,
                    static_cast<int64_t>(sh.N) * bands * kgroups};
    return true;
}

// The filter-resident kernel when the filter fits in LDS, else the
// filter-ring kernel.
hipError_t launch_sparse_fused(const SparseShape &sh, const float *x, const float *wt, float *y, const Decision &dec,
                               hipStream_t s, const Epilogue &epi) {
    using namespace fused;
    FusedPlan p;
    if (!fused_plan(sh, &p)) return launch_sparse_fring(sh, x, wt, y, dec, s, epi);
    FusedArgs a{};
    a.x = x;
    a.wt = wt;
    a.y = y;
    a.N = sh.N; a.C = sh.C; a.H = sh.H; a.W = sh.W; a.K = sh.K; a.P = sh.P; a.Ho = sh.Ho; a.Wo = sh.Wo;
    a.cs = p.cs;
    a.rg = kWaves / p.cs;
    a.bands = (sh.Ho + a.rg * p.th - 1) / (a.rg * p.th);
    a.Kp = (sh.K + kLanes - 1) / kLanes * kLanes;
    a.kgroups = p.wreg ? a.Kp / kLanes : 1;
    a.wide = a.kgroups > 1 || sh.tu.wide_loads == 1;
    a.dec = dec;
    a.epi = epi;
    switch (sh.R) {
    case 1: return launch_r1(a, p, s);
    case 3: return launch_r3(a, p, s);
    default: return launch_r5(a, p, s);
    }
}

}  // namespace isc
