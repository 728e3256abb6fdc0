// Posterior kernel instantiations for coordinate width 12 (padded d <= 12),
// Matern-5/2 models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_dx3(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<3, false>(a, st);
}
}  // namespace bo
