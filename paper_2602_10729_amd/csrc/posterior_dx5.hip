// Posterior kernel instantiations for coordinate width 20 (padded d <= 20).
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_dx5(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<5>(a, st);
}
}  // namespace bo
