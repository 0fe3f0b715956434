// AUTO's per-shape crossover between the zero-skipping path and the dense
// path (the dispatcher of Sec. "Sparse Convolution"'s ISC against the Fig. 3
// GEMM, decided by the measured sparsity of the input).
#include "isc_internal.hpp"

#include <cmath>

namespace isc {

// Interim reading until the per-kernel cost model is calibrated: filters of
// 3x3 and larger feed every nonzero input to many outputs and win from a
// sparsity of about 0.8; a 1x1 filter is a plain matrix product, which the
// matrix cores run far faster than one multiply-add per nonzero and map.
unsigned long long crossover_nnz_limit(const SparseShape &sh) {
    const double total = static_cast<double>(sh.N) * sh.C * sh.H * sh.W;
    const double s = sh.R * sh.S >= 9 ? 0.8 : 0.95;
    return static_cast<unsigned long long>(std::floor((1.0 - s) * total));
}

}  // namespace isc
