// Posterior kernel instantiations for coordinate width 28 (padded d <= 28),
// Matern-5/2 models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_dx7(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<7, false>(a, st);
}
}  // namespace bo
