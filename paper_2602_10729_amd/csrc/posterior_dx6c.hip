// Posterior kernel instantiations for coordinate width 24 (padded routing plus
// deployment groups <= 24), composite-kernel models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_comp_dx6(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<6, true>(a, st);
}
}  // namespace bo
