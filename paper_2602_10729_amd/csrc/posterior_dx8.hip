// Posterior kernel instantiations for coordinate width 32 (padded d <= 32).
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_dx8(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<8>(a, st);
}
}  // namespace bo
