// GP posterior of a batch of candidate points, one objective per launch.
//
// Paper: workflow step (ii) evaluates the acquisition on samples of the
// joint posterior of the GP surrogates; the posterior of an exact GP at x*
// is mu = k*^T alpha and Sigma = k(x*,x*) - v^T v with v = L^{-1} k*.
//
// One workgroup (8 waves, two per SIMD) owns a tile of NT points:
//   phase 1 (VALU): the cross-covariance tile K*^T [n_pad x NT] of the
//     ARD Matern-5/2 kernel, computed from lengthscale-scaled coordinates by
//     direct differences (no |a|^2 + |b|^2 - 2ab cancellation). Each wave
//     owns NT/8 candidates (coordinates in registers) and walks the training
//     points one per lane, prefetching the next point, so every LDS store is
//     a contiguous 256-byte run; mu = K* alpha is reduced with shuffles.
//     K*^T is stored column-major with a column stride of n_pad + 4 floats
//     (mod 32 banks: 4), which keeps the phase-2 16-byte reads conflict-free.
//   phase 2 (MFMA): V = L^{-1} K*^T over the lower 16x16 blocks only,
//     row block by row block. Waves take row blocks in a snake order so the
//     triangle is split evenly; each row block's V rows live only in the
//     MFMA accumulators and are squared into per-column sums at once
//     (q = 1 needs only |v|^2; q > 1 also needs the cross products of batch
//     members, which sit in the same 4-lane group of the accumulator and
//     are exchanged with DPP quad permutes).
//   The 16 inner indices of a block are split as k = 4g + kk between the
//     four 16-lane groups g and the four MFMA steps kk, so each lane's four
//     A operands are four consecutive columns of L^{-1} (pre-packed by the
//     fit: one 16-byte load, 1 KiB per block per wave) and its four B
//     operands are four consecutive rows of K*^T (one 16-byte LDS read).
// MFMA: v_mfma_f32_16x16x4f32, A[i][k] from lane i + 16k, B[k][j] from lane
// j + 16k, D[i][j] in lane j + 16(i/4), element i%4.
#include <hip/hip_runtime.h>

#include "bo_internal.h"

namespace bo {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

// Compile-time tuning of the posterior kernel (set with -D at build time).
#ifndef BO_POST_WAVES
#define BO_POST_WAVES 8      // waves per workgroup (2 per SIMD)
#endif
#ifndef BO_POST_PF
#define BO_POST_PF 4         // L^{-1} fragments in flight per wave
#endif
#ifndef BO_POST_NT_SMALL_N
#define BO_POST_NT_SMALL_N 32  // points per tile when n_pad <= 1024
#endif
constexpr int kWaves = BO_POST_WAVES;
constexpr int kThreads = 64 * kWaves;
constexpr int kPF = BO_POST_PF;

__device__ inline float matern52_f(float r2, float s) {
  const float r = __builtin_amdgcn_sqrtf(r2);
  // exp(-sqrt5 r) = 2^(-sqrt5 log2(e) r)
  constexpr float kNegSqrt5Log2e = static_cast<float>(-2.23606797749978969641 * 1.44269504088896340736);
  const float e = __builtin_amdgcn_exp2f(kNegSqrt5Log2e * r);
  const float poly = fmaf(r, 2.23606798f, fmaf(r2, 1.66666667f, 1.0f));
  return s * poly * e;
}

// Row block handled by a wave in round `it` (snake over the waves, so every
// wave's share of the lower triangle is the same up to one block).
__device__ inline int snake_block(int it, int wave) {
  return it * kWaves + ((it & 1) ? (kWaves - 1 - wave) : wave);
}

__device__ inline float quad_xor(float v, int x) {
  // DPP quad_perm: lane i of each group of 4 reads lane i ^ x.
  int iv = __float_as_int(v);
  int r;
  if (x == 1) r = __builtin_amdgcn_mov_dpp(iv, 0xB1, 0xF, 0xF, false);      // [1,0,3,2]
  else if (x == 2) r = __builtin_amdgcn_mov_dpp(iv, 0x4E, 0xF, 0xF, false); // [2,3,0,1]
  else r = __builtin_amdgcn_mov_dpp(iv, 0x1B, 0xF, 0xF, false);             // [3,2,1,0]
  return __int_as_float(r);
}

// Column stride of the K*^T tile in LDS: n_pad rounded to 32 floats plus 4,
// so the sixteen columns read by one 16-lane group start 4 banks apart.
__host__ __device__ inline int kt_stride(int n_pad) { return (n_pad + 31) / 32 * 32 + 4; }

// One 16x16 block pair: A fragment av, B fragments bv (one per 16-column
// block); MFMAs alternate between the column blocks so consecutive ones are
// independent.
template <int NCB>
__device__ inline void mfma_step(const float4 av, const float4 (&bv)[NCB], floatx4 (&acc)[NCB]) {
#pragma unroll
  for (int b = 0; b < NCB; ++b) acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av.x, bv[b].x, acc[b], 0, 0, 0);
#pragma unroll
  for (int b = 0; b < NCB; ++b) acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av.y, bv[b].y, acc[b], 0, 0, 0);
#pragma unroll
  for (int b = 0; b < NCB; ++b) acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av.z, bv[b].z, acc[b], 0, 0, 0);
#pragma unroll
  for (int b = 0; b < NCB; ++b) acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av.w, bv[b].w, acc[b], 0, 0, 0);
}

template <int NT, int DX4, int Q>
__global__ __launch_bounds__(kThreads) void k_posterior(PosteriorArgs a) {
  extern __shared__ float smem[];
  constexpr int NCB = NT / 16;          // 16-column blocks per tile
  constexpr int NX = (Q > 1) ? Q : 1;   // per-point partial slots (diag + xors)
  constexpr int CPW = NT / kWaves;      // candidates per wave in phase 1
  static_assert(CPW >= 1 && NT % kWaves == 0, "tile width vs waves");
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // wave index as a scalar: row-block control flow below stays uniform
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n_pad = a.nb * kBlk;
  const int ks = kt_stride(n_pad);
  float* Kt = smem;                                  // NT * ks, column-major
  float* red = smem + (size_t)NT * ks;               // kWaves * NT * NX
  float* mush = red + kWaves * NT * NX;              // NT
  float* kpp = mush + NT;                            // NT * 4 (prior cross-cov)
  const int64_t p0 = (int64_t)blockIdx.x * NT;

  // ---- phase 1: K*^T tile into LDS, mu -------------------------------------
  {
    float c[CPW][DX4 * 4];
    bool valid[CPW];
#pragma unroll
    for (int u = 0; u < CPW; ++u) {
      const int64_t p = p0 + wave * CPW + u;
      valid[u] = p < a.npts;
#pragma unroll
      for (int t = 0; t < DX4 * 4; ++t) c[u][t] = 0.f;
      if (valid[u]) {
        const float* cp = a.cand + p * a.d;
#pragma unroll
        for (int t = 0; t < DX4 * 4; ++t)
          if (t < a.d) c[u][t] = cp[t] * a.invls[t];
      }
    }
    float mu_part[CPW];
#pragma unroll
    for (int u = 0; u < CPW; ++u) mu_part[u] = 0.f;
    // training point `row` per lane; the next one is fetched ahead
    float4 xn[DX4];
    float aln = 0.f;
    if (lane < n_pad) {
      const float4* xr = reinterpret_cast<const float4*>(a.Xs + (size_t)lane * a.dx);
#pragma unroll
      for (int t4 = 0; t4 < DX4; ++t4) xn[t4] = xr[t4];
      aln = a.alpha[lane];
    }
    float* kcol = Kt + (size_t)(wave * CPW) * ks;
    for (int row0 = 0; row0 < n_pad; row0 += 64) {
      const int row = row0 + lane;
      float4 x[DX4];
#pragma unroll
      for (int t4 = 0; t4 < DX4; ++t4) x[t4] = xn[t4];
      const float al = aln;
      const int nrow = row + 64;
      if (nrow < n_pad) {
        const float4* xr = reinterpret_cast<const float4*>(a.Xs + (size_t)nrow * a.dx);
#pragma unroll
        for (int t4 = 0; t4 < DX4; ++t4) xn[t4] = xr[t4];
        aln = a.alpha[nrow];
      }
      if (row < n_pad) {
        const bool live = row < a.n;
#pragma unroll
        for (int u = 0; u < CPW; ++u) {
          float r2 = 0.f;
#pragma unroll
          for (int t4 = 0; t4 < DX4; ++t4) {
            const float d0 = c[u][4 * t4 + 0] - x[t4].x;
            const float d1 = c[u][4 * t4 + 1] - x[t4].y;
            const float d2 = c[u][4 * t4 + 2] - x[t4].z;
            const float d3 = c[u][4 * t4 + 3] - x[t4].w;
            r2 = fmaf(d0, d0, r2);
            r2 = fmaf(d1, d1, r2);
            r2 = fmaf(d2, d2, r2);
            r2 = fmaf(d3, d3, r2);
          }
          const float kv = (valid[u] && live) ? matern52_f(r2, a.s) : 0.f;
          mu_part[u] = fmaf(al, kv, mu_part[u]);
          kcol[(size_t)u * ks + row] = kv;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < CPW; ++u) {
      float v = mu_part[u];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
      if (lane == 0) mush[wave * CPW + u] = v;
    }
    if (Q > 1) {
      // prior covariance of each point with its batch mates (point ^ x),
      // one partner per lane
#pragma unroll
      for (int u = 0; u < CPW; ++u) {
        const int colu = wave * CPW + u;
        const int x = lane;
        if (x >= 1 && x < Q) {
          const int64_t pm = (p0 + colu) ^ x;
          float r2 = 0.f;
          if (valid[u] && pm < a.npts) {
            const float* cp = a.cand + pm * a.d;
#pragma unroll
            for (int t = 0; t < DX4 * 4; ++t)
              if (t < a.d) {
                const float dd = c[u][t] - cp[t] * a.invls[t];
                r2 = fmaf(dd, dd, r2);
              }
          }
          kpp[colu * 4 + x] = matern52_f(r2, a.s);
        }
      }
    }
  }
  __syncthreads();

  // ---- phase 2: V = L^{-1} K*^T on MFMA, squared on the fly ---------------
  float ss[NCB];
  float gx[NCB][NX];
#pragma unroll
  for (int b = 0; b < NCB; ++b) {
    ss[b] = 0.f;
#pragma unroll
    for (int x = 0; x < NX; ++x) gx[b][x] = 0.f;
  }
  const float4* Lp4 = reinterpret_cast<const float4*>(a.Lp);
  // B fragments: column (b*16 + lane%16), rows J*16 + 4*(lane/16) .. +3
  const float* Kb = Kt + (size_t)(lane & 15) * ks + 4 * (lane >> 4);
  const int bstride = 16 * ks;
  for (int it = 0;; ++it) {
    const int I = snake_block(it, wave);
    if (I >= a.nb) break;
    floatx4 acc[NCB];
#pragma unroll
    for (int b = 0; b < NCB; ++b) acc[b] = floatx4{0.f, 0.f, 0.f, 0.f};
    // row block I of L^{-1}: blocks (I, 0..I), 1 KiB each, consecutive.
    // A fragments run kPF blocks ahead, B fragments one block ahead; loads
    // past block I are clamped to I (in bounds, never consumed).
    const float4* Ablk = Lp4 + (size_t)I * (I + 1) / 2 * 64 + lane;
    const int nJ = I + 1;
    float4 ring[kPF];
#pragma unroll
    for (int u = 0; u < kPF; ++u) ring[u] = Ablk[(size_t)min(u, I) * 64];
    float4 bv[NCB];
#pragma unroll
    for (int b = 0; b < NCB; ++b) bv[b] = *reinterpret_cast<const float4*>(Kb + b * bstride);
    int J = 0;
    // Each step issues the loads for later steps first, then its eight
    // MFMAs; scheduling barriers keep the compiler from sinking the loads
    // next to their consumers (which would expose their latency).
    for (; J + kPF <= nJ; J += kPF) {
#pragma unroll
      for (int u = 0; u < kPF; ++u) {
        const float4 cur = ring[u];
        ring[u] = Ablk[(size_t)min(J + u + kPF, I) * 64];
        const int Jn = min(J + u + 1, I);
        float4 bn[NCB];
#pragma unroll
        for (int b = 0; b < NCB; ++b)
          bn[b] = *reinterpret_cast<const float4*>(Kb + b * bstride + Jn * 16);
        __builtin_amdgcn_sched_barrier(0);
        mfma_step<NCB>(cur, bv, acc);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int b = 0; b < NCB; ++b) bv[b] = bn[b];
      }
    }
#pragma unroll
    for (int u = 0; u < kPF; ++u) {
      if (J + u < nJ) {
        const int Jn = min(J + u + 1, I);
        float4 bn[NCB];
#pragma unroll
        for (int b = 0; b < NCB; ++b)
          bn[b] = *reinterpret_cast<const float4*>(Kb + b * bstride + Jn * 16);
        __builtin_amdgcn_sched_barrier(0);
        mfma_step<NCB>(ring[u], bv, acc);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int b = 0; b < NCB; ++b) bv[b] = bn[b];
      }
    }
#pragma unroll
    for (int b = 0; b < NCB; ++b) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float v = acc[b][r];
        ss[b] = fmaf(v, v, ss[b]);
        if (Q > 1) {
#pragma unroll
          for (int x = 1; x < NX; ++x) gx[b][x] = fmaf(v, quad_xor(v, x), gx[b][x]);
        }
      }
    }
  }
  // reduce over the four 16-lane row groups, then over waves in LDS
#pragma unroll
  for (int b = 0; b < NCB; ++b) {
    ss[b] += __shfl_xor(ss[b], 16);
    ss[b] += __shfl_xor(ss[b], 32);
#pragma unroll
    for (int x = 1; x < NX; ++x) {
      gx[b][x] += __shfl_xor(gx[b][x], 16);
      gx[b][x] += __shfl_xor(gx[b][x], 32);
    }
    if (lane < 16) {
      const int cc = b * 16 + lane;
      red[(wave * NT + cc) * NX + 0] = ss[b];
#pragma unroll
      for (int x = 1; x < NX; ++x) red[(wave * NT + cc) * NX + x] = gx[b][x];
    }
  }
  __syncthreads();

  // ---- epilogue -------------------------------------------------------------
  if (tid < NT) {
    const int64_t p = p0 + tid;
    const bool valid = p < a.npts;
    float tot[NX];
#pragma unroll
    for (int x = 0; x < NX; ++x) tot[x] = 0.f;
    for (int w = 0; w < kWaves; ++w)
#pragma unroll
      for (int x = 0; x < NX; ++x) tot[x] += red[(w * NT + tid) * NX + x];
    const float mu = mush[tid];
    const float var = a.s - tot[0];
    if (valid) {
      a.mu[p * a.m + a.k] = mu;
      a.sd[p * a.m + a.k] = __builtin_amdgcn_sqrtf(fmaxf(var, 0.f));
    }
    if (Q > 1) {
      // covariance row of this point (diagonal, then partner p ^ x) for the
      // batch owner; each thread rewrites only its own kpp slots
      kpp[tid * 4 + 0] = var;
#pragma unroll
      for (int x = 1; x < NX; ++x) kpp[tid * 4 + x] -= tot[x];
    }
  }
  if (Q > 1) {
    __syncthreads();
    constexpr int NB = NT / Q;
    if (tid < NB) {
      const int64_t bat = (int64_t)blockIdx.x * NB + tid;
      if (bat * Q < a.npts) {
        float S[Q][Q];
#pragma unroll
        for (int i = 0; i < Q; ++i)
#pragma unroll
          for (int j = 0; j < Q; ++j)
            S[i][j] = (i == j) ? kpp[(tid * Q + i) * 4 + 0] : kpp[(tid * Q + i) * 4 + (i ^ j)];
        float C[Q][Q];
#pragma unroll
        for (int i = 0; i < Q; ++i)
#pragma unroll
          for (int j = 0; j < Q; ++j) C[i][j] = 0.f;
        const float tol = 1e-10f * a.s;
#pragma unroll
        for (int j = 0; j < Q; ++j) {
          float pv = S[j][j];
#pragma unroll
          for (int t = 0; t < j; ++t) pv = fmaf(-C[j][t], C[j][t], pv);
          if (pv > tol) {
            const float cjj = __builtin_amdgcn_sqrtf(pv);
            C[j][j] = cjj;
            const float inv = 1.0f / cjj;
#pragma unroll
            for (int i = j + 1; i < Q; ++i) {
              float num = S[i][j];
#pragma unroll
              for (int t = 0; t < j; ++t) num = fmaf(-C[i][t], C[j][t], num);
              C[i][j] = num * inv;
            }
          }
        }
        constexpr int T = Q * (Q + 1) / 2;
        float* dst = a.chol + (bat * a.m + a.k) * T;
#pragma unroll
        for (int i = 0; i < Q; ++i)
#pragma unroll
          for (int j = 0; j <= i; ++j) dst[i * (i + 1) / 2 + j] = C[i][j];
      }
    }
  }
}

template <int NT, int DX4, int Q>
hipError_t launch_t(const PosteriorArgs& a, hipStream_t st) {
  const int n_pad = a.nb * kBlk;
  const size_t lds = sizeof(float) * ((size_t)NT * kt_stride(n_pad) +
                                      kWaves * NT * ((Q > 1) ? Q : 1) + NT + NT * 4);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_posterior<NT, DX4, Q>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       static_cast<int>(160 * 1024));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const unsigned grid = static_cast<unsigned>((a.npts + NT - 1) / NT);
  hipLaunchKernelGGL((k_posterior<NT, DX4, Q>), dim3(grid), dim3(kThreads), lds, st, a);
  return hipGetLastError();
}

template <int NT, int Q>
hipError_t launch_dx(const PosteriorArgs& a, hipStream_t st) {
  switch (a.dx / 4) {
    case 1: return launch_t<NT, 1, Q>(a, st);
    case 2: return launch_t<NT, 2, Q>(a, st);
    case 3: return launch_t<NT, 3, Q>(a, st);
    case 4: return launch_t<NT, 4, Q>(a, st);
    case 5: return launch_t<NT, 5, Q>(a, st);
    case 6: return launch_t<NT, 6, Q>(a, st);
    case 7: return launch_t<NT, 7, Q>(a, st);
    case 8: return launch_t<NT, 8, Q>(a, st);
    default: return hipErrorInvalidValue;
  }
}

template <int NT>
hipError_t launch_q(const PosteriorArgs& a, hipStream_t st) {
  switch (a.q) {
    case 1: return launch_dx<NT, 1>(a, st);
    case 2: return launch_dx<NT, 2>(a, st);
    case 4: return launch_dx<NT, 4>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

// Tile width: 32 points when K*^T fits LDS with room to spare, else 16.
int posterior_tile(int nb) { return (nb * kBlk <= 1024) ? BO_POST_NT_SMALL_N : 16; }

size_t posterior_lds_bytes(int nb, int q) {
  const int NT = posterior_tile(nb);
  return sizeof(float) * ((size_t)NT * kt_stride(nb * kBlk) + kWaves * NT * ((q > 1) ? q : 1) +
                          NT + NT * 4);
}

hipError_t launch_posterior(const PosteriorArgs& a, hipStream_t st) {
  if (a.npts <= 0) return hipSuccess;
  if (posterior_tile(a.nb) == 32) return launch_q<32>(a, st);
  return launch_q<16>(a, st);
  static_assert(BO_POST_NT_SMALL_N == 16 || BO_POST_NT_SMALL_N == 32, "tile width");
}

}  // namespace bo
