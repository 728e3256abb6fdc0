// Posterior kernel instantiations for coordinate width 12 (padded routing plus
// deployment groups <= 12), composite-kernel models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_comp_dx3(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<3, true>(a, st);
}
}  // namespace bo
