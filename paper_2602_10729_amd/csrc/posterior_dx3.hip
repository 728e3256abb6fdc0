// Posterior kernel instantiations for coordinate width 12 (padded d <= 12).
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_dx3(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<3>(a, st);
}
}  // namespace bo
