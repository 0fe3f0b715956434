// Filter-resident kernels for 3x3 filters (one translation unit per filter
// size, compiled in parallel); the kernel is in sparse_fused.hpp.
#define ISC_FUSED_INSTANTIATE
#include "sparse_fused.hpp"

namespace isc {
namespace fused {

hipError_t launch_r3(const FusedArgs &a, const FusedPlan &p, hipStream_t s) { return launch_fused_rs<3>(a, p, s); }

}  // namespace fused
}  // namespace isc
