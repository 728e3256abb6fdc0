// Device scratch of the scoring entry point that allocates nothing
// (bo_score_noalloc): one fixed array per device, holding a call's boxes and
// its posterior workspace (mean, standard deviation and batch factors).
//
// The array is a file-scope __device__ variable: every device the library
// runs on gets its own copy when the code object loads, and keeps it until
// the process ends. Host code never passes the array's name to a kernel (on
// the host it is only a stand-in symbol); it looks up the device address
// once per device, with that device current, and uses that address.
#include <hip/hip_runtime.h>

#include <mutex>

#include "bo_internal.h"

namespace bo {
namespace {

static __device__ __align__(256) float scratch[kNoallocScratchFloats];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxScratchDevices] = {};

}  // namespace

bo_status noalloc_scratch(int dev, float** out) {
  *out = nullptr;
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(BO_ERR_DEVICE, "bo_score_noalloc: device index out of range");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return hip_fail(e, "bo_score_noalloc: current device");
    if (cur != dev) return fail(BO_ERR_DEVICE, "bo_score_noalloc: scratch looked up off its device");
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "bo_score_noalloc: scratch address");
    g_scratch_ptr[dev] = static_cast<float*>(p);
  }
  *out = g_scratch_ptr[dev];
  return BO_OK;
}

}  // namespace bo
