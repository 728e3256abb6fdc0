// Power-of-two scaling of kernel values before their fp16 hi/lo split,
// shared by the kernels that feed kernel values to the fp16 matrix cores.
#pragma once

#include <hip/hip_runtime.h>

namespace bo {
// Power-of-two scale of one candidate's kernel values before their fp16
// hi/lo split. Every |k(x*, x_i)| is at most sqrt(k(x*, x*) k(x_i, x_i)) (a
// covariance), so with `bound` at least that and bound = f 2^E (f in
// [0.5, 1)) the values times 2^(14 - E) are at most 2^14: far below fp16's
// largest finite value (65504). Every scaled value of at least 2^-3 (2^-17
// of the bound) then splits into halves that are normal fp16 numbers (or an
// exact zero low half); smaller ones lose at most 2^-25 absolute, 2^-39 of
// the bound. ksc = 2^(14 - E) scales, kinv = 2^(E - 14) undoes it
// (both exact); a bound that is not finite and positive gives NaN for both,
// so the candidate's results read NaN.
struct KvScale {
  float ksc, kinv;
};
__device__ inline KvScale kv_split_scale(float bound) {
  if (!(bound > 0.f) || !(bound < __builtin_huge_valf()))
    return KvScale{__builtin_nanf(""), __builtin_nanf("")};
  const int E = __builtin_amdgcn_frexp_expf(bound);
  return KvScale{__builtin_amdgcn_ldexpf(1.0f, 14 - E), __builtin_amdgcn_ldexpf(1.0f, E - 14)};
}

}  // namespace bo
