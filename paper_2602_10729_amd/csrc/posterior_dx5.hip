// Posterior kernel instantiations for coordinate width 20 (padded d <= 20),
// Matern-5/2 models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_dx5(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<5, false>(a, st);
}
}  // namespace bo
