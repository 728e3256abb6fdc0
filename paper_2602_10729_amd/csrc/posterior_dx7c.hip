// Posterior kernel instantiations for coordinate width 28 (padded routing plus
// deployment groups <= 28), composite-kernel models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_comp_dx7(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<7, true>(a, st);
}
}  // namespace bo
