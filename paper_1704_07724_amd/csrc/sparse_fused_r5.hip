// Filter-resident kernels for 5x5 filters (one translation unit per filter
// size, compiled in parallel); the kernel is in sparse_fused.hpp.
#define ISC_FUSED_INSTANTIATE
#include "sparse_fused.hpp"

namespace isc {
namespace fused {

hipError_t launch_r5(const FusedArgs &a, const FusedPlan &p, hipStream_t s) { return launch_fused_rs<5>(a, p, s); }

}  // namespace fused
}  // namespace isc
