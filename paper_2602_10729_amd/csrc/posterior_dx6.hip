// Posterior kernel instantiations for coordinate width 24 (padded d <= 24),
// Matern-5/2 models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_dx6(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<6, false>(a, st);
}
}  // namespace bo
