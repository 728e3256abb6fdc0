// Posterior kernel instantiations for coordinate width 8 (padded d <= 8),
// Matern-5/2 models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_dx2(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<2, false>(a, st);
}
}  // namespace bo
