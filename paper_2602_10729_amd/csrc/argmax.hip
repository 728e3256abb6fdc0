// Argmax over the candidates' acquisition values.
//
// Paper: workflow step (ii) selects the maximiser of the acquisition as the
// next configuration to evaluate. Semantics: lowest index among equal
// maxima, NaN never wins, -1 when nothing qualifies.
//
// Each (value, index) is packed into one 64-bit key whose unsigned order is
// the wanted order: the high word maps the float's bits to an order-
// preserving unsigned code, the low word is 0xFFFFFFFF - index so that a
// smaller index compares larger. One coalesced grid-stride pass reduces
// keys per wave with shuffles, per block in LDS, and a single 64-bit atomic
// max per block lands in the caller's index cell, which a 1-thread launch
// initialised to 0 (no valid key is 0) and a final 1-thread launch decodes.
#include <hip/hip_runtime.h>

#include "bo_internal.h"

namespace bo {
namespace {

__device__ inline unsigned long long pack_key(float v, int64_t i) {
  if (v != v) return 0ull;
  const unsigned u = __float_as_uint(v);
  const unsigned ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<unsigned long long>(ord) << 32) |
         static_cast<unsigned long long>(0xFFFFFFFFu - static_cast<unsigned>(i));
}

__global__ void k_argmax_init(int64_t* index) {
  *reinterpret_cast<unsigned long long*>(index) = 0ull;
}

__global__ __launch_bounds__(256) void k_argmax_reduce(const float* __restrict__ v,
                                                       int64_t M, int64_t* index) {
  __shared__ unsigned long long wbest[4];
  unsigned long long best = 0ull;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < M; i += stride) {
    const unsigned long long k = pack_key(v[i], i);
    best = k > best ? k : best;
  }
  for (int off = 32; off > 0; off >>= 1) {
    const unsigned long long o = __shfl_xor(best, off);
    best = o > best ? o : best;
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) wbest[w] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long b = wbest[0];
    for (int i = 1; i < 4; ++i) b = wbest[i] > b ? wbest[i] : b;
    if (b != 0ull) atomicMax(reinterpret_cast<unsigned long long*>(index), b);
  }
}

__global__ void k_argmax_final(const float* __restrict__ v, int64_t* index, float* value) {
  const unsigned long long k = *reinterpret_cast<unsigned long long*>(index);
  if (k == 0ull) {
    *index = -1;
    *value = __builtin_nanf("");
  } else {
    const int64_t i = static_cast<int64_t>(0xFFFFFFFFu - static_cast<unsigned>(k & 0xFFFFFFFFull));
    *index = i;
    *value = v[i];
  }
}

}  // namespace

hipError_t launch_argmax(const float* v, int64_t M, int64_t* index, float* value,
                         hipStream_t st) {
  hipLaunchKernelGGL(k_argmax_init, dim3(1), dim3(1), 0, st, index);
  if (M > 0) {
    int64_t blocks = (M + 256 * 8 - 1) / (256 * 8);
    if (blocks > 2048) blocks = 2048;
    hipLaunchKernelGGL(k_argmax_reduce, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                       st, v, M, index);
  }
  hipLaunchKernelGGL(k_argmax_final, dim3(1), dim3(1), 0, st, v, index, value);
  return hipGetLastError();
}

}  // namespace bo
