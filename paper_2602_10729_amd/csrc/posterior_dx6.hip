// Posterior kernel instantiations for coordinate width 24 (padded d <= 24).
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_dx6(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<6>(a, st);
}
}  // namespace bo
