// Weight-gradient kernels for 5x5 filters (one translation unit per filter
// size, compiled in parallel); the kernel is in sparse_dw.hpp.
#define ISC_DW_INSTANTIATE
#include "sparse_dw.hpp"

namespace isc {
namespace dwk {

hipError_t launch_r5(const DwArgs &a, const DwPlan &p, hipStream_t s) { return launch_dw_rs<5>(a, p, s); }

}  // namespace dwk
}  // namespace isc
