// Posterior kernel instantiations for coordinate width 4 (padded d <= 4),
// Matern-5/2 models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_dx1(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<1, false>(a, st);
}
}  // namespace bo
