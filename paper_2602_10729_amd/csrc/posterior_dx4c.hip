// Posterior kernel instantiations for coordinate width 16 (padded routing plus
// deployment groups <= 16), composite-kernel models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_comp_dx4(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<4, true>(a, st);
}
}  // namespace bo
