// Posterior kernel instantiations for coordinate width 32 (padded routing plus
// deployment groups <= 32), composite-kernel models.
#include "posterior_kernel.h"

namespace bo {
hipError_t launch_posterior_comp_dx8(const PosteriorArgs& a, hipStream_t st) {
  return launch_for_dx<8, true>(a, st);
}
}  // namespace bo
