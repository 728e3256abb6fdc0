// Device characterisation: achievable peaks that the roofline fractions of
// the scoring kernels are read against (alongside the datasheet figures).
//
//   BO_PEAK_VALU_FMA   — independent v_fma_f32 chains, no packed math
//                        (lane-ops/s; one FMA = one lane-op)
//   BO_PEAK_VALU_CLAMP — the EHVI inner pattern (sub, med3, fma) per lane
//                        (lane-ops/s)
//   BO_PEAK_MFMA_F32   — independent v_mfma_f32_16x16x4f32 chains (flop/s)
//   BO_PEAK_HBM_COPY   — float4 streaming copy of a large buffer (bytes/s,
//                        read + write)
//   BO_PEAK_MFMA_F16   — independent v_mfma_f32_16x16x32_f16 chains (flop/s)
// Each runs a fixed amount of work over the whole chip (2048 workgroups of
// 256 threads) on the given stream and times it with HIP events.
#include <hip/hip_runtime.h>

#include "bo_internal.h"

namespace bo {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
constexpr int kGrid = 2048;
constexpr int kBlock = 256;

__global__ __launch_bounds__(kBlock) void k_valu_fma(float* out, int iters, float a, float b) {
  float x[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = static_cast<float>(threadIdx.x + i);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = fmaf(x[i], a, b);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) s += x[i];
  if (s == 1.2345f) out[blockIdx.x * kBlock + threadIdx.x] = s;   // keep the work
}

__global__ __launch_bounds__(kBlock) void k_valu_clamp(float* out, int iters, float lo, float w) {
  float y[8];
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) y[i] = static_cast<float>(threadIdx.x + i) * 1e-3f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
      const float t0 = __builtin_amdgcn_fmed3f(y[i] - lo, 0.0f, w);
      const float t1 = __builtin_amdgcn_fmed3f(y[i + 1] - lo, 0.0f, w);
      acc = fmaf(t0, t1, acc);
    }
    lo += 1e-7f;
  }
  if (acc == 1.2345f) out[blockIdx.x * kBlock + threadIdx.x] = acc;
}

constexpr int kChains = 8;   // independent accumulators per wave

__global__ __launch_bounds__(kBlock) void k_mfma(float* out, int iters) {
  floatx4 acc[kChains];
#pragma unroll
  for (int i = 0; i < kChains; ++i) acc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
  const float a = static_cast<float>(threadIdx.x) * 1e-3f;
  const float b = 1.0f - a;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kChains; ++i)
      acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[i], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kChains; ++i) s += acc[i][0] + acc[i][1] + acc[i][2] + acc[i][3];
  if (s == 1.2345f) out[blockIdx.x * kBlock + threadIdx.x] = s;
}

__global__ __launch_bounds__(kBlock) void k_mfma_f16(float* out, int iters) {
  floatx4 acc[kChains];
#pragma unroll
  for (int i = 0; i < kChains; ++i) acc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
  halfx8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = static_cast<_Float16>(static_cast<float>(threadIdx.x) * 1e-3f + i);
    b[i] = static_cast<_Float16>(1.0f - i * 1e-2f);
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kChains; ++i)
      acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, acc[i], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kChains; ++i) s += acc[i][0] + acc[i][1] + acc[i][2] + acc[i][3];
  if (s == 1.2345f) out[blockIdx.x * kBlock + threadIdx.x] = s;
}

__global__ __launch_bounds__(kBlock) void k_copy(const float4* __restrict__ src,
                                                 float4* __restrict__ dst, int64_t n4) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n4; i += stride) dst[i] = src[i];
}

}  // namespace

hipError_t measure_peak(int what, int64_t iters, double* rate, hipStream_t st) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  float* scratch = nullptr;
  float4* buf = nullptr;
  const int64_t copy_bytes = (int64_t)1 << 30;
  if (e == hipSuccess) e = hipMalloc(&scratch, sizeof(float) * kGrid * kBlock);
  if (e == hipSuccess && what == BO_PEAK_HBM_COPY) e = hipMalloc(&buf, 2 * copy_bytes);
  double work = 0.0;
  const int it = static_cast<int>(iters);
  for (int rep = 0; rep < 2 && e == hipSuccess; ++rep) {   // first pass warms up
    e = hipEventRecord(e0, st);
    if (e != hipSuccess) break;
    switch (what) {
      case BO_PEAK_VALU_FMA:
        hipLaunchKernelGGL(k_valu_fma, dim3(kGrid), dim3(kBlock), 0, st, scratch, it, 0.999f, 1e-3f);
        work = (double)kGrid * kBlock * 8.0 * it;
        break;
      case BO_PEAK_VALU_CLAMP:
        hipLaunchKernelGGL(k_valu_clamp, dim3(kGrid), dim3(kBlock), 0, st, scratch, it, 0.1f, 0.5f);
        work = (double)kGrid * kBlock * 4.0 * 5.0 * it;   // 4 x (2 sub, 2 med3, 1 fma)
        break;
      case BO_PEAK_MFMA_F32:
        hipLaunchKernelGGL(k_mfma, dim3(kGrid), dim3(kBlock), 0, st, scratch, it);
        work = (double)kGrid * (kBlock / 64) * kChains * 2048.0 * it;
        break;
      case BO_PEAK_MFMA_F16:
        hipLaunchKernelGGL(k_mfma_f16, dim3(kGrid), dim3(kBlock), 0, st, scratch, it);
        work = (double)kGrid * (kBlock / 64) * kChains * 16384.0 * it;
        break;
      case BO_PEAK_HBM_COPY: {
        const int64_t n4 = copy_bytes / 16;
        hipLaunchKernelGGL(k_copy, dim3(kGrid * 4), dim3(kBlock), 0, st, buf, buf + n4, n4);
        work = 2.0 * copy_bytes;
        break;
      }
      default:
        e = hipErrorInvalidValue;
    }
    if (e == hipSuccess) e = hipGetLastError();
    if (e == hipSuccess) e = hipEventRecord(e1, st);
    if (e == hipSuccess) e = hipEventSynchronize(e1);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
    if (e == hipSuccess) *rate = work / (ms * 1e-3);
  }
  (void)hipFree(scratch);
  (void)hipFree(buf);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  return e;
}

}  // namespace bo
