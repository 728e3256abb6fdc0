// Posterior kernel instantiations for coordinate width 16 (padded d <= 16),
// Matern-5/2 models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_dx4(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<4, false>(a, st);
}
}  // namespace bo
