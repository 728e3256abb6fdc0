// Posterior kernel instantiations for coordinate width 20 (padded routing plus
// deployment groups <= 20), composite-kernel models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_comp_dx5(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<5, true>(a, st);
}
}  // namespace bo
