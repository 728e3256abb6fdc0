// Posterior kernel instantiations for coordinate width 32 (padded d <= 32),
// Matern-5/2 models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_dx8(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<8, false>(a, st);
}
}  // namespace bo
