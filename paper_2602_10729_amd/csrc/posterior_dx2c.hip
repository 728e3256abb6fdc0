// Posterior kernel instantiations for coordinate width 8 (padded routing plus
// deployment groups <= 8), composite-kernel models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_comp_dx2(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<2, true>(a, st);
}
}  // namespace bo
