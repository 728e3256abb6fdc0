// GP posterior of a batch of candidate points: dispatch over the coordinate
// width to the kernel instantiations (the kernel itself, and what it
// computes, is described in posterior_kernel.h).
#include "posterior_kernel.h"

namespace bo {

size_t posterior_lds_bytes(int nb, int q) {
  (void)nb;
  return sizeof(float) * lds_floats(BO_POST_NT, 8, q);   // widest coordinate stride
}

int64_t posterior_frag_blocks(int nb) { return frag_row_start(nb) + 1; }

hipError_t launch_posterior(const PosteriorArgs& a, hipStream_t st) {
  if (a.npts <= 0) return hipSuccess;
  if (a.dr > 0) {
    switch (a.dx / 4) {
      case 2: return launch_posterior_comp_dx2(a, st);
      case 3: return launch_posterior_comp_dx3(a, st);
      case 4: return launch_posterior_comp_dx4(a, st);
      case 5: return launch_posterior_comp_dx5(a, st);
      case 6: return launch_posterior_comp_dx6(a, st);
      case 7: return launch_posterior_comp_dx7(a, st);
      case 8: return launch_posterior_comp_dx8(a, st);
      default: return hipErrorInvalidValue;
    }
  }
  switch (a.dx / 4) {
    case 1: return launch_posterior_dx1(a, st);
    case 2: return launch_posterior_dx2(a, st);
    case 3: return launch_posterior_dx3(a, st);
    case 4: return launch_posterior_dx4(a, st);
    case 5: return launch_posterior_dx5(a, st);
    case 6: return launch_posterior_dx6(a, st);
    case 7: return launch_posterior_dx7(a, st);
    case 8: return launch_posterior_dx8(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace bo

