// Filter-ring kernels for 5x5 filters (one translation unit per filter size,
// compiled in parallel); the kernel is in sparse_fring.hpp.
#define ISC_FRING_INSTANTIATE
#include "sparse_fring.hpp"

namespace isc {
namespace fring {

hipError_t launch_r5(const FringArgs &a, const TileChoice &tc, hipStream_t s) {
    return launch_fring_rs<5>(a, tc, s);
}

}  // namespace fring
}  // namespace isc
