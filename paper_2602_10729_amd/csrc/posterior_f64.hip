// GP posterior of a batch of candidate points in fp64 (models fitted with
// bo_fit_f64 / bo_fit_composite_f64), one objective per launch.
//
// Paper: implementation section (the GP kernels run in double precision);
// the posterior of an exact GP at x* is mu = k*^T alpha and
// Sigma = k(x*, x*) - v^T v with v = L^{-1} k*.
//
// Everything a candidate's posterior needs is fp64 here: the scaled
// differences (c_t - x_t) / l_t from the fp32 inputs, the kernel values, mu,
// and V = L^{-1} K*^T on the fp64 matrix cores (v_mfma_f64_16x16x4f64, fp64
// accumulation), so the variance keeps its relative accuracy where
// sigma^2 = k(x, x) - |v|^2 cancels (candidates near the data, long
// lengthscales learned by the marginal likelihood). mu, sigma and the batch
// factor are rounded to fp32 once, for the acquisition.
//
// One workgroup (8 waves) owns a tile of NT = 16 NCB points and forms V
// left-looking over 32-row blocks J of K*^T (eight MFMA k-steps of 4 rows):
// every block is produced once into LDS (double-buffered, one barrier per
// block) while the matrix cores add W[I][J] K*^T[J] into the accumulators of
// the 16-row blocks I >= 2J that each wave owns (RBW slots per wave, snake
// order). All n rows of V stay in the accumulators, so nothing is produced
// twice. The training rows of block J + 2 are staged in LDS while block J + 1
// is produced.
//
// Fragments of v_mfma_f64_16x16x4f64: A[i][k] from lane i + 16k, B[k][j] from
// lane j + 16k, D[i][j] in lane j + 16(i%4), element i/4. Only the pairing of
// A's and B's k and D's columns (lane % 16) are used.
#include <hip/hip_runtime.h>

#include <cmath>

#include "bo_internal.h"

namespace bo {
namespace {

typedef double doublex4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kJ = 32;          // rows of K*^T per block (eight k-steps of 4)
constexpr int kKs = 34;         // LDS stride of one column of a produced block (doubles)

__device__ inline double m52d(double r2) {
  const double r = sqrt(r2);
  const double c = 2.23606797749978969641;   // sqrt(5)
  return (1.0 + c * r + (5.0 / 3.0) * r2) * exp(-c * r);
}

__device__ inline double m32d(double r2) {
  const double r = sqrt(r2);
  const double c = 1.73205080756887729353;   // sqrt(3)
  return (1.0 + c * r) * exp(-c * r);
}

__device__ __forceinline__ double quad_xor_d(double v, int x) {
  // DPP quad_perm on both halves: lane i of each group of 4 reads lane i ^ x
  const int lo = __builtin_bit_cast(int2, v).x, hi = __builtin_bit_cast(int2, v).y;
  int rl, rh;
  if (x == 1) {
    rl = __builtin_amdgcn_mov_dpp(lo, 0xB1, 0xF, 0xF, false);
    rh = __builtin_amdgcn_mov_dpp(hi, 0xB1, 0xF, 0xF, false);
  } else if (x == 2) {
    rl = __builtin_amdgcn_mov_dpp(lo, 0x4E, 0xF, 0xF, false);
    rh = __builtin_amdgcn_mov_dpp(hi, 0x4E, 0xF, 0xF, false);
  } else {
    rl = __builtin_amdgcn_mov_dpp(lo, 0x1B, 0xF, 0xF, false);
    rh = __builtin_amdgcn_mov_dpp(hi, 0x1B, 0xF, 0xF, false);
  }
  return __builtin_bit_cast(double, int2{rl, rh});
}

// Index of packed block (I, 0): row block I holds the blocks J = 0 .. I/2.
__host__ __device__ __forceinline__ int f64_row_start(int I) {
  const int t = I >> 1;
  return (I & 1) ? (t + 1) * (t + 1) : t * (t + 1);
}

template <int RBW, int NCB, int Q, bool COMP>
__global__ __launch_bounds__(kThreads) void k_posterior_f64(PosteriorArgs a) {
  constexpr int NT = 16 * NCB;          // points per tile
  constexpr int PER = kJ * NT / kThreads;   // kernel values per thread per block (1 or 2)
  constexpr int NX = (Q > 1) ? Q : 1;
  static_assert(PER >= 1 && kJ * NT == PER * kThreads, "whole blocks per step");
  __shared__ __align__(16) double kb[2][NT * kKs];      // produced blocks [col][pos(row)]
  // the tile's candidates (fp64 of fp32), coordinate-major: the lanes of a
  // wave read consecutive candidates of one coordinate (no bank conflicts)
  __shared__ double cs[BO_MAX_D][NT];
  __shared__ double ils[BO_MAX_D];                      // 1 / lengthscale (fp64)
  __shared__ float xst[2][kJ][BO_MAX_D];                // staged training rows
  __shared__ double wst[2][kJ];                         // composite: their preference weights
  __shared__ double wsh[NT];                            // composite: the candidates' weights
  __shared__ double red[kWaves][NT][NX];                // per-wave column sums
  __shared__ double mup[kJ * NT / NT][NT];              // mu partials [row thread][column]
  __shared__ double kpp[NT][4];                         // q > 1: prior covariance with batch mates

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int d = a.d, n = a.n, nb = a.nb;
  const int nbj = (nb + 1) / 2;
  const int64_t p0 = (int64_t)blockIdx.x * NT;
  const double s = a.s;

  // candidates, inverse lengthscales, and (composite) the candidates' weights
  for (int e = tid; e < NT * d; e += kThreads) {
    const int c = e / d, t = e % d;
    const int64_t p = p0 + c;
    cs[t][c] = (p < a.npts) ? static_cast<double>(a.cand[p * d + t]) : 0.0;
  }
  for (int t = tid; t < d; t += kThreads) ils[t] = a.ils64[t];
  __syncthreads();
  if (COMP && tid < NT) {
    double e = 0.0;
    for (int t = a.dr; t < d; ++t) e = fma(static_cast<double>(a.pref[t - a.dr]), cs[t][tid], e);
    wsh[tid] = exp(e);
  }

  // stage the training rows of block jb (rows past n read zero)
  auto stage = [&](int jb) {
    for (int e = tid; e < kJ * d; e += kThreads) {
      const int r = e / d, t = e % d;
      const int row = jb * kJ + r;
      xst[jb & 1][r][t] = (row < n) ? a.Xraw[(int64_t)row * d + t] : 0.f;
    }
  };
  auto stage_weights = [&](int jb) {
    if (COMP && tid < kJ) {
      double e = 0.0;
      for (int t = a.dr; t < d; ++t)
        e = fma(static_cast<double>(a.pref[t - a.dr]), static_cast<double>(xst[jb & 1][tid][t]), e);
      wst[jb & 1][tid] = exp(e);
    }
  };
  // produce block jb into kb[jb & 1]: thread tid makes rows (tid + kThreads e) / NT
  // for column (tid + kThreads e) % NT, stored at position (row % 4) * 8 + row / 4
  double mu_acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) mu_acc[e] = 0.0;
  auto produce = [&](int jb) {
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int idx = tid + kThreads * e;
      const int col = idx % NT, r = idx / NT;
      const int row = jb * kJ + r;
      double ra = 0.0, rc = 0.0;        // plain: all in ra; composite: routing / deployment
      for (int t = 0; t < d; ++t) {
        const double df = (cs[t][col] - static_cast<double>(xst[jb & 1][r][t])) * ils[t];
        if (COMP && t >= a.dr) rc = fma(df, df, rc);
        else ra = fma(df, df, ra);
      }
      double kv;
      if constexpr (COMP) {
        const double k5 = m52d(ra), k3 = m32d(rc);
        kv = s * k5 + static_cast<double>(a.s_dep) * wsh[col] * wst[jb & 1][r] * k3 +
             static_cast<double>(a.s_int) * k5 * k3;
      } else {
        kv = s * m52d(ra);
      }
      if (row >= n) kv = 0.0;
      else mu_acc[e] = fma(a.alpha64[row], kv, mu_acc[e]);
      kb[jb & 1][col * kKs + (r % 4) * 8 + r / 4] = kv;
    }
  };

  // q > 1: prior covariance of each point with its batch mates
  if (Q > 1 && tid < NT * 4) {
    const int c = tid / 4, x = tid % 4;
    double v = 0.0;
    if (x >= 1 && x < Q) {
      const int cm = c ^ x;
      double ra = 0.0, rc = 0.0;
      for (int t = 0; t < d; ++t) {
        const double df = (cs[t][c] - cs[t][cm]) * ils[t];
        if (COMP && t >= a.dr) rc = fma(df, df, rc);
        else ra = fma(df, df, ra);
      }
      if constexpr (COMP) {
        const double k5 = m52d(ra), k3 = m32d(rc);
        v = s * k5 + static_cast<double>(a.s_dep) * wsh[c] * wsh[cm] * k3 +
            static_cast<double>(a.s_int) * k5 * k3;
      } else {
        v = s * m52d(ra);
      }
    }
    kpp[c][x] = v;
  }

  // slots of this wave: row block base_t + (t even ? wave : 7 - wave)
  int slotI[RBW];
#pragma unroll
  for (int t = 0; t < RBW; ++t) slotI[t] = 8 * t + ((t & 1) ? (kWaves - 1 - wave) : wave);
  doublex4 acc[RBW][NCB];
#pragma unroll
  for (int t = 0; t < RBW; ++t)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[t][cb] = doublex4{0.0, 0.0, 0.0, 0.0};

  stage(0);
  if (nbj > 1) stage(1);
  __syncthreads();
  stage_weights(0);
  if (nbj > 1) stage_weights(1);
  __syncthreads();
  produce(0);

  for (int J = 0; J < nbj; ++J) {
    __syncthreads();            // block J visible; every wave is done with block J - 1
    if (J + 1 < nbj) produce(J + 1);
    if (J + 2 < nbj) stage(J + 2);      // into xst[J & 1], read last by produce(J)
    // B fragments of block J: column 16 cb + lane % 16, rows 4 kk + lane / 16
    double bfr[NCB][8];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      const double* src = &kb[J & 1][(16 * cb + (lane & 15)) * kKs + (lane >> 4) * 8];
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) bfr[cb][kk] = src[kk];
    }
#pragma unroll
    for (int t = 0; t < RBW; ++t) {
      const int I = slotI[t];
      if (I < nb && 2 * J <= I) {
        // A fragment of block (I, J): W[16 I + lane % 16][32 J + 4 kk + lane / 16]
        const double* ap = a.Lp64 + ((int64_t)(f64_row_start(I) + J) * 64 + lane) * 8;
        double afr[8];
#pragma unroll
        for (int kk = 0; kk < 8; kk += 2) {
          const double2 v = *reinterpret_cast<const double2*>(ap + kk);
          afr[kk] = v.x;
          afr[kk + 1] = v.y;
        }
#pragma unroll
        for (int kk = 0; kk < 8; ++kk)
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb)
            acc[t][cb] = __builtin_amdgcn_mfma_f64_16x16x4f64(afr[kk], bfr[cb][kk], acc[t][cb], 0, 0, 0);
      }
    }
    __syncthreads();            // staged rows of block J + 2 visible
    if (J + 2 < nbj) stage_weights(J + 2);
  }

  // |v|^2 per column (and cross products with batch mates), over the lanes of
  // a column, then over waves
  double ss[NCB][NX];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int x = 0; x < NX; ++x) ss[cb][x] = 0.0;
#pragma unroll
  for (int t = 0; t < RBW; ++t)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const double v = acc[t][cb][i];
        ss[cb][0] = fma(v, v, ss[cb][0]);
#pragma unroll
        for (int x = 1; x < NX; ++x) ss[cb][x] = fma(v, quad_xor_d(v, x), ss[cb][x]);
      }
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int x = 0; x < NX; ++x) {
      double v = ss[cb][x];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (lane < 16) red[wave][16 * cb + lane][x] = v;
    }
  // mu partials: thread tid holds column tid % NT for rows (tid + kThreads e) / NT
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int idx = tid + kThreads * e;
    mup[idx / NT][idx % NT] = mu_acc[e];
  }
  __syncthreads();

  if (tid < NT) {
    const int64_t p = p0 + tid;
    double tot[NX];
#pragma unroll
    for (int x = 0; x < NX; ++x) tot[x] = 0.0;
    for (int w = 0; w < kWaves; ++w)
#pragma unroll
      for (int x = 0; x < NX; ++x) tot[x] += red[w][tid][x];
    double mu = 0.0;
    for (int r = 0; r < kJ; ++r) mu += mup[r][tid];
    double prior = s;
    if constexpr (COMP) {
      const double w = wsh[tid];
      prior = s + static_cast<double>(a.s_dep) * w * w + static_cast<double>(a.s_int);
    }
    const double var = prior - tot[0];
    if (p < a.npts) {
      a.mu[p * a.mu_ps] = static_cast<float>(mu);
      // clamp at zero; a NaN variance stays NaN
      a.sd[p * a.sd_ps] = static_cast<float>(sqrt(var < 0.0 ? 0.0 : var));
    }
    if (Q > 1) {
      kpp[tid][0] = var;
#pragma unroll
      for (int x = 1; x < NX; ++x) kpp[tid][x] -= tot[x];
    }
  }
  if (Q > 1) {
    __syncthreads();
    constexpr int NBAT = NT / Q;
    if (tid < NBAT) {
      const int64_t bat = (int64_t)blockIdx.x * NBAT + tid;
      if (bat * Q < a.npts) {
        double S[Q][Q], L[Q][Q];
#pragma unroll
        for (int i = 0; i < Q; ++i)
#pragma unroll
          for (int j = 0; j < Q; ++j) {
            S[i][j] = (i == j) ? kpp[tid * Q + i][0] : kpp[tid * Q + i][i ^ j];
            L[i][j] = 0.0;
          }
        // the same PSD rule as the fp32 path: a Schur pivot <= 1e-10 times the
        // prior scale zeroes its column
        const double tol = 1e-10 * (COMP ? s + static_cast<double>(a.s_dep) + static_cast<double>(a.s_int) : s);
#pragma unroll
        for (int j = 0; j < Q; ++j) {
          double pv = S[j][j];
#pragma unroll
          for (int t = 0; t < j; ++t) pv -= L[j][t] * L[j][t];
          if (pv > tol) {
            const double ljj = sqrt(pv);
            L[j][j] = ljj;
#pragma unroll
            for (int i = j + 1; i < Q; ++i) {
              double num = S[i][j];
#pragma unroll
              for (int t = 0; t < j; ++t) num -= L[i][t] * L[j][t];
              L[i][j] = num / ljj;
            }
          } else if (pv != pv) {
            L[j][j] = pv;
          }
        }
        constexpr int T = Q * (Q + 1) / 2;
        float* dst = a.chol + bat * T;
#pragma unroll
        for (int i = 0; i < Q; ++i)
#pragma unroll
          for (int j = 0; j <= i; ++j) dst[i * (i + 1) / 2 + j] = static_cast<float>(L[i][j]);
      }
    }
  }
}

template <int RBW, int NCB, bool COMP>
hipError_t launch_rb(const PosteriorArgs& a, hipStream_t st) {
  const int NT = 16 * NCB;
  const unsigned grid = static_cast<unsigned>((a.npts + NT - 1) / NT);
  switch (a.q) {
    case 1: hipLaunchKernelGGL((k_posterior_f64<RBW, NCB, 1, COMP>), dim3(grid), dim3(kThreads), 0, st, a); break;
    case 2: hipLaunchKernelGGL((k_posterior_f64<RBW, NCB, 2, COMP>), dim3(grid), dim3(kThreads), 0, st, a); break;
    case 4: hipLaunchKernelGGL((k_posterior_f64<RBW, NCB, 4, COMP>), dim3(grid), dim3(kThreads), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <bool COMP>
hipError_t launch_comp(const PosteriorArgs& a, hipStream_t st) {
  // every row block of V in the accumulators: 8 waves x RBW slots of 16 rows
  if (a.nb <= 16) return launch_rb<2, 2, COMP>(a, st);
  if (a.nb <= 32) return launch_rb<4, 2, COMP>(a, st);
  if (a.nb <= 64) return launch_rb<8, 2, COMP>(a, st);
  if (a.nb <= 128) return launch_rb<16, 1, COMP>(a, st);
  return hipErrorInvalidValue;
}

// Pack W = L^{-1} (fp64, [m][nf][nf], lower) as A fragments of
// v_mfma_f64_16x16x4f64: block (I, J) of 16 rows x 32 columns at index
// f64_row_start(I) + J, lane l holding W[16 I + l%16][32 J + 4 kk + l/16] for
// kk = 0..7 (zero above the diagonal and past n), 4 KiB per block.
__global__ __launch_bounds__(256) void k_pack_f64(const double* __restrict__ W, int64_t n, int nf,
                                                  int64_t nblk, double* __restrict__ Lp) {
  const int k = blockIdx.y;
  const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (g >= nblk * 64) return;
  const int64_t blk = g / 64;
  const int lane = static_cast<int>(g % 64);
  int64_t t = static_cast<int64_t>((sqrt(4.0 * blk + 1.0) - 1.0) * 0.5);
  while ((t + 1) * (t + 2) <= blk) ++t;
  while (t * (t + 1) > blk) --t;
  int I, J;
  if (blk >= (t + 1) * (t + 1)) {
    I = static_cast<int>(2 * t + 1);
    J = static_cast<int>(blk - (t + 1) * (t + 1));
  } else {
    I = static_cast<int>(2 * t);
    J = static_cast<int>(blk - t * (t + 1));
  }
  const int64_t row = (int64_t)I * 16 + lane % 16;
  const double* Wk = W + (int64_t)k * nf * nf;
  double* dst = Lp + ((int64_t)k * nblk + blk) * 512 + lane * 8;
  for (int kk = 0; kk < 8; ++kk) {
    const int64_t col = (int64_t)J * 32 + 4 * kk + lane / 16;
    dst[kk] = (row < n && col <= row) ? Wk[row * nf + col] : 0.0;
  }
}

}  // namespace

int64_t posterior_f64_blocks(int nb) { return f64_row_start(nb); }

hipError_t launch_pack_f64(const double* W, int64_t n, int m, int nf, int nb, double* Lp64,
                           hipStream_t st) {
  const int64_t nblk = f64_row_start(nb);
  const unsigned gx = static_cast<unsigned>((nblk * 64 + 255) / 256);
  hipLaunchKernelGGL(k_pack_f64, dim3(gx, m), dim3(256), 0, st, W, n, nf, nblk, Lp64);
  return hipGetLastError();
}

hipError_t launch_posterior_f64(const PosteriorArgs& a, hipStream_t st) {
  if (a.npts <= 0) return hipSuccess;
  if (a.d > BO_MAX_D) return hipErrorInvalidValue;
  return a.dr > 0 ? launch_comp<true>(a, st) : launch_comp<false>(a, st);
}

}  // namespace bo
