// Weight-gradient kernel (sparse_dw.hpp): the plan, the ordered sum of the
// ranges and the launch.
#include "sparse_dw.hpp"

#include <algorithm>
#include <cstdlib>

namespace isc {
namespace dwk {
namespace {

// dw[e] = sum over ranges of part[range][e], ranges in order.
__global__ __launch_bounds__(256)
void dw_reduce_kernel(const float *__restrict__ part, int splits, int64_t n, float *__restrict__ dw) {
    const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (e >= n) return;
    float s = 0.0f;
    for (int i = 0; i < splits; ++i) s += part[static_cast<int64_t>(i) * n + e];
    dw[e] = s;
}

// Tile rows and maps per lane (measured on every workload layer):
//  - 3x3 filters: one-row tiles, two maps per lane;
//  - 5x5 and 1x1 filters: two-row tiles (each scanned nonzero feeds two
//    output rows), two maps per lane -- one when K > 64 with 5x5 filters,
//    which keeps three channels per wavefront instead of one.
// A caller's tuning maps_per_lane (1, 2, 4) and rows (1, 2) override the
// choice (four maps per lane only with one-row 16-column tiles, two rows
// only with one or two maps per lane).
int dw_th(const SparseShape &sh) {
    const int t = sh.tu.rows;
    if (t == 1 || t == 2) return t;
    return sh.R == 3 ? 1 : 2;
}

int dw_kpl(const SparseShape &sh, int th) {
    const int k = sh.tu.maps_per_lane;
    if ((k == 1 || k == 2) || (k == 4 && th == 1 && sh.Wo <= 16)) return k;
    return sh.R == 5 && sh.K > kLanes ? 1 : 2;
}
int dw_tw(int Wo) { return Wo <= 16 ? 16 : 28; }

bool dw_plan(const SparseShape &sh, DwPlan *p) {
    if (sh.T != 1 || sh.R != sh.S || !(sh.R == 1 || sh.R == 3 || sh.R == 5)) return false;
    p->th = dw_th(sh);
    p->kpl = dw_kpl(sh, p->th);
    p->ch = dw_ch_for(sh.R, p->kpl, p->th);
    p->tw = p->th == 2 ? 16 : dw_tw(sh.Wo);
    p->TWr = std::min(p->tw, sh.Wo);
    p->ctiles = (sh.Wo + p->TWr - 1) / p->TWr;
    p->bands = (sh.Ho + p->th - 1) / p->th;
    p->kgroups = (sh.K + kLanes * p->kpl - 1) / (kLanes * p->kpl);
    const int cgroups = (sh.C + p->ch - 1) / p->ch;
    p->cquads = (cgroups + kDwWaves - 1) / kDwWaves;
    const int64_t ntiles = static_cast<int64_t>(sh.N) * p->bands * p->ctiles;
    if (ntiles > (1ll << 30)) return false;
    p->ntiles = static_cast<int>(ntiles);
    const int64_t base = static_cast<int64_t>(p->kgroups) * p->cquads;
    int64_t splits = std::max<int64_t>(1, std::min<int64_t>(ntiles, (kDwMinGroups + base - 1) / base));
    p->per = static_cast<int>((ntiles + splits - 1) / splits);
    p->splits = static_cast<int>((ntiles + p->per - 1) / p->per);
    return base * p->splits < (1ll << 31);
}

}  // namespace
}  // namespace dwk

bool sparse_dw_applies(const SparseShape &sh) {
    dwk::DwPlan p;
    return dwk::dw_plan(sh, &p);
}

// The largest partial-sum buffer of any tile the overrides may force, so
// that one workspace size holds for every plan.
size_t sparse_dw_workspace_floats(const SparseShape &sh) {
    size_t most = 0;
    for (int th : {1, 2})
        for (int kpl : {1, 2, 4}) {
            SparseShape v = sh;
            v.tu = isc_tuning{};
            v.tu.rows = th;
            v.tu.maps_per_lane = kpl;
            dwk::DwPlan p;
            if (dwk::dw_plan(v, &p)) most = std::max(most, static_cast<size_t>(p.splits) * sh.K * sh.C * sh.R * sh.S);
        }
    return most;
}

hipError_t launch_sparse_dw(const SparseShape &sh, const float *x, const float *dy, float *dw, float *part,
                            hipStream_t s) {
    using namespace dwk;
    DwPlan p;
    if (!dw_plan(sh, &p)) return hipErrorInvalidValue;
    DwArgs a{};
    a.x = x;
    a.dy = dy;
    a.part = part;
    a.N = sh.N; a.C = sh.C; a.H = sh.H; a.W = sh.W; a.K = sh.K; a.P = sh.P; a.Ho = sh.Ho; a.Wo = sh.Wo;
    a.TWr = p.TWr;
    a.ctiles = p.ctiles;
    a.bands = p.bands;
    a.cquads = p.cquads;
    a.splits = p.splits;
    a.per = p.per;
    a.ntiles = p.ntiles;
    hipError_t e = sh.R == 1 ? launch_r1(a, p, s) : sh.R == 3 ? launch_r3(a, p, s) : launch_r5(a, p, s);
    if (e != hipSuccess) return e;
    const int64_t n = static_cast<int64_t>(sh.K) * sh.C * sh.R * sh.S;
    dw_reduce_kernel<<<static_cast<unsigned>((n + 255) / 256), 256, 0, s>>>(part, p.splits, n, dw);
    return hipGetLastError();
}

}  // namespace isc
