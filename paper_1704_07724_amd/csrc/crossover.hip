// AUTO's per-shape crossover between the zero-skipping path and the dense
// path: the dispatcher of the paper's ISC (Sec. "Sparse Convolution")
// against the matrix-multiplication formulation of Fig. 3, decided by the
// measured sparsity of the input.  The paper's CPU experiments put the
// crossover near a sparsity of 0.9 (Abstract); on this GPU it depends on the
// shape: from below 0.5 (LeNet conv2, 5x5 filters at batch 256) to never
// (1x1 filters at batch 128, which the matrix cores run faster at any
// sparsity).
//
// Both paths' times are modelled from the plan the launch would run.  The
// sparse path's time is linear in the input's density d = 1 - sparsity:
//   t_sparse(d) = c0 + c1 * F_scan + c2 * d * F_nz + c3 * F_chain
// with, per wavefront-channel of the plan (Wc of them), the window's
// positions (F_scan: the scan's tests, the ring's LDS traffic), the window's
// nonzeros times their work (F_nz: scalar dispatch plus taps times maps per
// lane in multiply-adds), and the channels each wavefront walks in sequence
// (F_chain: memory latency per channel on small grids; for the
// register-weight kernel times the rounds of resident workgroups).  The coefficients
// of each kernel family (the register-weight kernel's per filter size) were
// fitted to the sparse path measured on every workload and Tab. 2 shape at
// sparsities 0.5 to 0.99 (5-9 % rms); the
// dense path's model is in dense_conv.hip.  The limit handed to the device
// is the largest nonzero count whose modelled sparse time does not exceed
// the modelled dense time; the device compares integers only.
#include "isc_internal.hpp"

#include <algorithm>
#include <cmath>

namespace isc {
namespace {

struct Fit {
    double c0, c_scan, c_nz, c_chain;  // ms; features scaled by 1e-9 (1e-3 for the chain)
};

constexpr Fit kRingFit{0.07996214, 1.82930381, 1.78868403, 0.0};
// the register-weight kernel per filter size (1x1, 3x3, 5x5: its only
// ones), whose chain feature counts the rounds of resident workgroups
constexpr Fit kRegFit1{0.020774588, 1.0001204, 0.45244511, 0.30880721};
constexpr Fit kRegFit3{0.023252027, 1.112875, 0.44553699, 0.46230413};
constexpr Fit kRegFit5{0.019268499, 2.1330448, 1.0296948, 0.91803993};
// its workgroups per CU: eight wavefronts each, 60-66 VGPRs for 1x1 and 3x3
// filters (eight wavefronts per SIMD, the 33 KB of reduction tiles four
// times over), 80-98 for 5x5 (five per SIMD)
inline int reg_workgroups_per_cu(int R) { return R == 5 ? 2 : 4; }
constexpr Fit kResidentFit{0.01847326, 0.0, 1.77078063, 1.41836285};

}  // namespace

long long crossover_nnz_limit(const SparseShape &sh) {
    const int64_t total = static_cast<int64_t>(sh.N) * sh.C * sh.H * sh.W;
    isc_plan p{};
    if (!sparse_fused_plan_info(sh, &p)) {
        // kernels over compacted lists: no model, the paper's 0.9
        return static_cast<long long>(std::floor(0.1 * static_cast<double>(total)));
    }
    const Fit &freg = sh.R == 1 ? kRegFit1 : (sh.R == 3 ? kRegFit3 : kRegFit5);
    const Fit &f = p.kernel == ISC_KERNEL_FUSED_RING ? kRingFit : (p.kernel == ISC_KERNEL_FUSED_REG ? freg : kResidentFit);
    const double wc = static_cast<double>(p.workgroups) * p.waves * sh.C / std::max(1, p.phases);
    const int wrows = (p.rows - 1) * sh.T + sh.R, wcols = (p.cols - 1) * sh.T + sh.S;
    const double pw = static_cast<double>(wrows) * wcols;
    const double pin = static_cast<double>(std::min(wrows, sh.H)) * std::min(wcols, sh.W);
    const double useful = static_cast<double>(std::min(p.rows, sh.Ho)) * std::min(p.cols, sh.Wo);
    const double taps = std::min<double>(sh.R * sh.S, useful * sh.R * sh.S / pin);
    const int kpl = std::max(1, p.maps_per_lane);
    double scan;
    if (p.kernel == ISC_KERNEL_FUSED_RING) {
        const double wbytes = 4.0 * sh.R * sh.S * 64 * kpl;
        scan = wc * (pw * 1.65 + wbytes / 128.0 * (1.0 + 1.0 / std::max(1, p.waves))) * 1e-9;
    } else {
        scan = wc * pw * 1e-9;
    }
    // channels each wavefront walks in sequence; for the register-weight
    // kernel, whose wavefronts wait on their own chain of loads and scans,
    // times the rounds of resident workgroups the grid takes
    double chain = static_cast<double>(sh.C) / std::max(1, p.phases) * 1e-3;
    if (p.kernel == ISC_KERNEL_FUSED_REG)
        chain *= std::ceil(static_cast<double>(p.workgroups) / (256.0 * reg_workgroups_per_cu(sh.R)));
    const double fixed = f.c0 + f.c_scan * scan + f.c_chain * chain;
    const double per_density = f.c_nz * wc * pin * (10.0 + taps * kpl) * 1e-9;
    const double dense = dense_time_model(sh.K, static_cast<int64_t>(sh.N) * sh.Ho * sh.Wo,
                                          static_cast<int64_t>(sh.C) * sh.R * sh.S);
    if (!(per_density > 0.0)) return dense >= fixed ? static_cast<long long>(total) : -1;
    const double dstar = (dense - fixed) / per_density;  // density at which the two meet
    // a crossover past 0.95 sparsity counts as none: keeping the choice open
    // (the count, and the gated launch of the path not taken) costs more on
    // every call than the sparse path could save on the rare inputs past it
    // (Tab. 2's inception 4a.1 at batch 128: modelled crossover 0.97-0.99,
    // measured none up to 0.99; AUTO 18 % over the dense path at 0.9 while
    // it kept the choice)
    if (dstar < 0.05) return -1;
    if (dstar >= 1.0) return static_cast<long long>(total);
    return static_cast<long long>(std::floor(dstar * static_cast<double>(total)));
}

}  // namespace isc
