// Monte-Carlo (q)EHVI over a disjoint box decomposition.
//
// Paper: "Constrained qNEHVI" paragraph — the acquisition is the expected
// hypervolume improvement over samples of the joint posterior, estimated by
// Monte-Carlo integration, optionally restricted to feasible samples. With
// the region the front does not dominate split into disjoint boxes
// [lo, lo + w):
//   HVI(y)  = sum_c prod_k clamp(y_k - lo_ck, 0, w_ck)
//   qHVI(Y) = sum_{J != {}} (-1)^{|J|+1} sum_c prod_k min_{a in J} clamp(y_ak - lo_ck, 0, w_ck)
// (the clamp is monotone, so the minimum over batch members commutes with it).
//
// Feasibility (the constrained form): the constraints bound the objectives
// themselves, y_k >= t_k on the maximised objectives, and a sample (a batch
// member) counts only where all of them hold. An infeasible member's first
// objective is replaced by -inf: every clamp of it is then 0, so each box
// product, and each subset term that contains the member, vanishes — the
// same as multiplying those terms by the member's indicator.
//
// Mapping: one lane per candidate batch; the S base samples and the boxes
// are the same for every lane, so they sit in LDS and every read is a
// broadcast. For q > 1 a box that only one member reaches (on any lane and
// sample of the chunk) adds that member's own extent product; the other
// subset terms are exact zeros. Samples are processed in chunks held in registers and each box
// is read once per chunk, which leaves a branch-free VALU loop of
// 2m + (m-1) + 1 ops per (sample, box) for q = 1. No cross-lane reduction is
// needed: a lane owns all S x boxes terms of its candidate.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "bo_internal.h"

namespace bo {
namespace {

constexpr int kThreads = 256;

__device__ inline float clamp_ext(float y, float lo, float w) {
  return __builtin_amdgcn_fmed3f(y - lo, 0.0f, w);
}

// Member feasibility: all objectives at or above their thresholds.
template <int MO>
__device__ __forceinline__ float mask_infeasible(const float (&y)[MO], const EhviArgs& a) {
  bool ok = true;
#pragma unroll
  for (int k = 0; k < MO; ++k) ok = ok && (y[k] >= a.lower[k]);
  return ok ? y[0] : -__builtin_inff();
}

template <int MO, int SC, bool CONS>
__global__ __launch_bounds__(kThreads) void k_ehvi_q1(EhviArgs a) {
  extern __shared__ float sm[];
  float* zs = sm;                                   // [S][MO]
  float* bx = sm + a.S * MO;                        // [nbox][2*MO]
  for (int i = threadIdx.x; i < a.S * MO; i += kThreads) zs[i] = a.Z[i];
  for (int i = threadIdx.x; i < a.nbox * 2 * MO; i += kThreads) bx[i] = a.boxes[i];
  __syncthreads();
  const int64_t b = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const bool valid = b < a.nbat;
  float mu[MO], sd[MO];
  bool nan_in = false;      // a NaN posterior gives a NaN acquisition
#pragma unroll
  for (int k = 0; k < MO; ++k) {
    mu[k] = valid ? a.mu[b * a.mu_ps + k * a.mu_ks] : 0.f;
    sd[k] = valid ? a.sd[b * a.sd_ps + k * a.sd_ks] : 0.f;
    nan_in = nan_in || (mu[k] != mu[k]) || (sd[k] != sd[k]);
  }
  float acc = 0.f;
  for (int s0 = 0; s0 < a.S; s0 += SC) {
    float y[SC][MO];
#pragma unroll
    for (int j = 0; j < SC; ++j)
#pragma unroll
      for (int k = 0; k < MO; ++k) {
        const int s = s0 + j;
        const int sl = (s < a.S) ? s : (a.S - 1);
        // samples past S get -inf: every extent clamps to 0
        y[j][k] = (s < a.S) ? fmaf(sd[k], zs[sl * MO + k], mu[k]) : -__builtin_inff();
      }
    if constexpr (CONS) {
#pragma unroll
      for (int j = 0; j < SC; ++j) y[j][0] = mask_infeasible<MO>(y[j], a);
    }
    for (int c = 0; c < a.nbox; ++c) {
      float lo[MO], w[MO];
#pragma unroll
      for (int k = 0; k < MO; ++k) {
        lo[k] = bx[c * 2 * MO + k];
        w[k] = bx[c * 2 * MO + MO + k];
      }
#pragma unroll
      for (int j = 0; j < SC; ++j) {
        float t = clamp_ext(y[j][0], lo[0], w[0]);
#pragma unroll
        for (int k = 1; k < MO; ++k) t *= clamp_ext(y[j][k], lo[k], w[k]);
        acc += t;
      }
    }
  }
  if (valid) a.ehvi[b] = nan_in ? __builtin_nanf("") : acc / static_cast<float>(a.S);
}

// q-batch version: lane owns a batch of Q points; y_s[a][k] is sampled with
// the lower factor of objective k, then the 2^Q - 1 member subsets are
// expanded by inclusion-exclusion per box. Batches are few (131,072 at the
// q = 4 workload: two waves per SIMD at one lane each), so the four waves of
// a workgroup share its 64 batches and split the samples; their partial sums
// are added in LDS in wave order.
constexpr int kQWaves = kThreads / 64;
template <int MO, int Q, int SC, bool CONS>
__global__ __launch_bounds__(kThreads) void k_ehvi_q(EhviArgs a) {
  extern __shared__ float sm[];
  constexpr int T = Q * (Q + 1) / 2;
  constexpr int NS = (1 << Q);
  float* zs = sm;                                   // [S][Q][MO]
  float* bx = sm + a.S * Q * MO;                    // [nbox][2*MO]
  for (int i = threadIdx.x; i < a.S * Q * MO; i += kThreads) zs[i] = a.Z[i];
  for (int i = threadIdx.x; i < a.nbox * 2 * MO; i += kThreads) bx[i] = a.boxes[i];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t b = (int64_t)blockIdx.x * 64 + lane;
  const bool valid = b < a.nbat;
  // this wave's samples: a quarter of S, in whole chunks of SC
  const int sw = (a.S + kQWaves * SC - 1) / (kQWaves * SC) * SC;
  const int sbeg = wave * sw, send = min(a.S, sbeg + sw);
  float mu[Q][MO];
  float C[MO][T];
  bool nan_in = false;      // a NaN posterior gives a NaN acquisition
#pragma unroll
  for (int i = 0; i < Q; ++i)
#pragma unroll
    for (int k = 0; k < MO; ++k) {
      mu[i][k] = valid ? a.mu[(b * Q + i) * a.mu_ps + k * a.mu_ks] : 0.f;
      nan_in = nan_in || (mu[i][k] != mu[i][k]);
    }
#pragma unroll
  for (int k = 0; k < MO; ++k)
#pragma unroll
    for (int e = 0; e < T; ++e) {
      C[k][e] = valid ? a.chol[(k * a.nbat + b) * T + e] : 0.f;
      nan_in = nan_in || (C[k][e] != C[k][e]);
    }

  float acc_pos = 0.f, acc_neg = 0.f;
  for (int s0 = sbeg; s0 < send; s0 += SC) {
    float y[SC][Q][MO];
#pragma unroll
    for (int j = 0; j < SC; ++j) {
      const int s = s0 + j;
      const int sl = (s < send) ? s : (send - 1);
#pragma unroll
      for (int k = 0; k < MO; ++k)
#pragma unroll
        for (int i = 0; i < Q; ++i) {
          float v = mu[i][k];
#pragma unroll
          for (int t = 0; t <= i; ++t) v = fmaf(C[k][i * (i + 1) / 2 + t], zs[(sl * Q + t) * MO + k], v);
          y[j][i][k] = (s < send) ? v : -__builtin_inff();
        }
      if constexpr (CONS) {
#pragma unroll
        for (int i = 0; i < Q; ++i) y[j][i][0] = mask_infeasible<MO>(y[j][i], a);
      }
    }
    // per sample, the batch's best value in each objective: a box whose
    // lower corner no member exceeds in some objective adds exactly zero
    float ymax[SC][MO];
#pragma unroll
    for (int j = 0; j < SC; ++j)
#pragma unroll
      for (int k = 0; k < MO; ++k) {
        float v = y[j][0][k];
#pragma unroll
        for (int i = 1; i < Q; ++i) v = fmaxf(v, y[j][i][k]);
        ymax[j][k] = v;
      }
    for (int c = 0; c < a.nbox; ++c) {
      float lo[MO], w[MO];
#pragma unroll
      for (int k = 0; k < MO; ++k) {
        lo[k] = bx[c * 2 * MO + k];
        w[k] = bx[c * 2 * MO + MO + k];
      }
      bool live = false;
#pragma unroll
      for (int j = 0; j < SC; ++j) {
        bool nz = true;
#pragma unroll
        for (int k = 0; k < MO; ++k) nz = nz && (ymax[j][k] > lo[k]);
        live = live || nz;
      }
      if (__ballot(live) == 0) continue;   // the whole wave would add zeros
      // the members that reach the box (above its lower corner in every
      // objective) on some lane and sample of the chunk; a member subset with
      // any other member adds exactly zero. Mostly one member reaches a box:
      // then only its own extent product is formed (the same sum, the other
      // terms being zeros)
      int rmask = 0;
#pragma unroll
      for (int i = 0; i < Q; ++i) {
        bool r = false;
#pragma unroll
        for (int j = 0; j < SC; ++j) {
          bool rj = true;
#pragma unroll
          for (int k = 0; k < MO; ++k) rj = rj && (y[j][i][k] > lo[k]);
          r = r || rj;
        }
        if (__ballot(r) != 0) rmask |= 1 << i;
      }
      if (rmask == 0) continue;
      if ((rmask & (rmask - 1)) == 0) {
#pragma unroll
        for (int i = 0; i < Q; ++i) {
          if (rmask == (1 << i)) {
#pragma unroll
            for (int j = 0; j < SC; ++j) {
              float t = clamp_ext(y[j][i][0], lo[0], w[0]);
#pragma unroll
              for (int k = 1; k < MO; ++k) t *= clamp_ext(y[j][i][k], lo[k], w[k]);
              acc_pos += t;
            }
          }
        }
        continue;
      }
#pragma unroll
      for (int j = 0; j < SC; ++j) {
        float ext[NS][MO];
#pragma unroll
        for (int i = 0; i < Q; ++i)
#pragma unroll
          for (int k = 0; k < MO; ++k) ext[1 << i][k] = clamp_ext(y[j][i][k], lo[k], w[k]);
#pragma unroll
        for (int mask = 1; mask < NS; ++mask) {
          const int low = mask & (-mask);
          if (mask != low) {
#pragma unroll
            for (int k = 0; k < MO; ++k) ext[mask][k] = fminf(ext[mask ^ low][k], ext[low][k]);
          }
          float t = ext[mask][0];
#pragma unroll
          for (int k = 1; k < MO; ++k) t *= ext[mask][k];
          if (__builtin_popcount(mask) & 1) acc_pos += t;
          else acc_neg += t;
        }
      }
    }
  }
  // the waves' partial sums, added in wave order (the samples' LDS is done)
  __syncthreads();
  float* part = sm;                                 // [kQWaves][64]
  part[wave * 64 + lane] = acc_pos - acc_neg;
  __syncthreads();
  if (wave == 0) {
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < kQWaves; ++w) tot += part[w * 64 + lane];
    if (valid) a.ehvi[b] = nan_in ? __builtin_nanf("") : tot / static_cast<float>(a.S);
  }
}

// Launch with the dynamic-LDS limit raised for that kernel (set on every
// launch, so that it holds on whichever device is current).
template <typename K>
hipError_t launch_k(K kern, unsigned grid, size_t lds, hipStream_t st, const EhviArgs& a) {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kThreads), lds, st, a);
  return hipGetLastError();
}

template <int MO, bool CONS>
hipError_t launch_mo(const EhviArgs& a, hipStream_t st) {
  // q = 1: a lane per candidate; q > 1: a workgroup per 64 batches
  const int per = (a.q == 1) ? kThreads : 64;
  const unsigned grid = static_cast<unsigned>((a.nbat + per - 1) / per);
  // (q > 1: at least the waves' partial sums, which reuse the space at the end)
  const size_t lds = sizeof(float) * std::max<size_t>((size_t)a.S * a.q * MO + (size_t)a.nbox * 2 * MO,
                                                      a.q > 1 ? kThreads : 0);
  switch (a.q) {
    case 1: return launch_k(&k_ehvi_q1<MO, 16, CONS>, grid, lds, st, a);
    case 2: return launch_k(&k_ehvi_q<MO, 2, 4, CONS>, grid, lds, st, a);
    case 4: return launch_k(&k_ehvi_q<MO, 4, 2, CONS>, grid, lds, st, a);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

size_t ehvi_lds_bytes(int S, int q, int m, int nbox) {
  return sizeof(float) * ((size_t)S * q * m + (size_t)nbox * 2 * m);
}

hipError_t launch_ehvi(const EhviArgs& a, hipStream_t st) {
  if (a.nbat <= 0) return hipSuccess;
  if (a.m == 2) return a.constrained ? launch_mo<2, true>(a, st) : launch_mo<2, false>(a, st);
  if (a.m == 3) return a.constrained ? launch_mo<3, true>(a, st) : launch_mo<3, false>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace bo
