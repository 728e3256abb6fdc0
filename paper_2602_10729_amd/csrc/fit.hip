// GP conditioning on the device, fp64 (off the scoring loop).
//
// Paper: workflow step (i), "Surrogate model fitting", with the ARD
// Matern-5/2 covariance in a scale kernel (implementation section). Exact
// conditioning of a Gaussian-noise GP needs the Cholesky factor of
// K = k(X, X) + eta I; the scoring path consumes L^{-1} (so the per-candidate
// triangular solve becomes a triangular matrix product on MFMA) and
// alpha = K^{-1} y.
//
// The fit is O(n^3) once per BO iteration against O(n^2) per candidate, so it
// runs in fp64 here: the fp32 scoring path then inherits factors rounded
// once, and its whole error budget goes to the scoring arithmetic.
//
// Blocked right-looking Cholesky with 64x64 blocks, three launches per block
// column:
//   potrf: factor the diagonal block in LDS and invert it (one workgroup per
//          objective);
//   trsm:  panel blocks below the diagonal times the inverse's transpose;
//   syrk:  trailing update of every lower block (ib >= jb' > jb).
// The inverse W = L^{-1} is built column block by column block: one
// workgroup per block column walks down it, W_ij = -D_i^{-1} sum_t L_it W_tj.
#include <hip/hip_runtime.h>

#include <cmath>

#include "bo_internal.h"

namespace bo {
namespace {

constexpr int B = kFitBlk;          // 64
constexpr int LDP = B + 1;          // padded LDS row (doubles)

__device__ inline double matern52_d(double r2, double s) {
  const double r = sqrt(r2);
  const double c = 2.23606797749978969641;   // sqrt(5)
  return s * (1.0 + c * r + (5.0 / 3.0) * r2) * exp(-c * r);
}

__global__ void k_gram(const float* __restrict__ X, int64_t n, int d, int nf,
                       const double* __restrict__ ls, const double* __restrict__ os,
                       const double* __restrict__ noise, double* __restrict__ A) {
  const int k = blockIdx.z;
  const int i = blockIdx.y * 16 + threadIdx.y;
  const int j = blockIdx.x * 16 + threadIdx.x;
  if (i >= nf || j >= nf) return;
  double v;
  if (i < n && j < n) {
    double r2 = 0.0;
    for (int t = 0; t < d; ++t) {
      const double diff = (static_cast<double>(X[(int64_t)i * d + t]) -
                           static_cast<double>(X[(int64_t)j * d + t])) / ls[k * d + t];
      r2 += diff * diff;
    }
    v = matern52_d(r2, os[k]);
    if (i == j) v += noise[k];
  } else {
    v = (i == j) ? 1.0 : 0.0;
  }
  A[((int64_t)k * nf + i) * nf + j] = v;
}

// Factor the diagonal block jb of every objective in LDS, write L_jj (lower,
// zeros above) back and its inverse to Dinv.
__global__ __launch_bounds__(256) void k_potrf(double* __restrict__ A,
                                               double* __restrict__ Dinv, int nf,
                                               int jb, int* __restrict__ flag) {
  __shared__ double a[B][LDP];
  __shared__ double x[B][LDP];
  __shared__ int bad;
  const int k = blockIdx.x;
  const int tid = threadIdx.x;
  double* Ak = A + (int64_t)k * nf * nf;
  const int o = jb * B;
  for (int e = tid; e < B * B; e += 256) {
    const int i = e / B, c = e % B;
    a[i][c] = Ak[(int64_t)(o + i) * nf + o + c];
  }
  if (tid == 0) bad = 0;
  __syncthreads();
  for (int j = 0; j < B; ++j) {
    if (tid == 0) {
      const double p = a[j][j];
      if (!(p > 0.0) || !isfinite(p)) {
        bad = 1;
        a[j][j] = 1.0;
      } else {
        a[j][j] = sqrt(p);
      }
    }
    __syncthreads();
    const double djj = a[j][j];
    for (int i = j + 1 + tid; i < B; i += 256) a[i][j] /= djj;
    __syncthreads();
    const int w = B - j - 1;
    for (int e = tid; e < w * w; e += 256) {
      const int i = j + 1 + e / w, c = j + 1 + e % w;
      if (c <= i) a[i][c] -= a[i][j] * a[c][j];
    }
    __syncthreads();
  }
  // inverse of the lower block: column c solves L x = e_c by substitution
  if (tid < B) {
    const int c = tid;
    for (int i = 0; i < B; ++i) {
      if (i < c) { x[i][c] = 0.0; continue; }
      double acc = (i == c) ? 1.0 : 0.0;
      for (int t = c; t < i; ++t) acc -= a[i][t] * x[t][c];
      x[i][c] = acc / a[i][i];
    }
  }
  __syncthreads();
  double* Dk = Dinv + ((int64_t)k * (nf / B) + jb) * B * B;
  for (int e = tid; e < B * B; e += 256) {
    const int i = e / B, c = e % B;
    Ak[(int64_t)(o + i) * nf + o + c] = (c <= i) ? a[i][c] : 0.0;
    Dk[e] = x[i][c];
  }
  if (tid == 0 && bad) atomicOr(flag, 1);
}

// 64x64x64 product helper: out[i][c] (4x4 per thread) = sum_t P[i][t] * Q[c][t].
__device__ inline void gemm_nt_64(const double (*P)[LDP], const double (*Q)[LDP],
                                  double acc[4][4], int ty, int tx) {
  for (int t = 0; t < B; ++t) {
    double pv[4], qv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) pv[r] = P[ty * 4 + r][t];
#pragma unroll
    for (int c = 0; c < 4; ++c) qv[c] = Q[tx * 4 + c][t];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[r][c] = fma(pv[r], qv[c], acc[r][c]);
  }
}

// Panel: A[ib][jb] <- A[ib][jb] * Dinv_jb^T for ib > jb.
__global__ __launch_bounds__(256) void k_trsm(double* __restrict__ A,
                                              const double* __restrict__ Dinv,
                                              int nf, int jb) {
  __shared__ double p[B][LDP];
  __shared__ double q[B][LDP];
  const int k = blockIdx.y;
  const int ib = jb + 1 + blockIdx.x;
  const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
  double* Ak = A + (int64_t)k * nf * nf;
  const double* Dk = Dinv + ((int64_t)k * (nf / B) + jb) * B * B;
  for (int e = tid; e < B * B; e += 256) {
    const int i = e / B, c = e % B;
    p[i][c] = Ak[(int64_t)(ib * B + i) * nf + jb * B + c];
    q[i][c] = Dk[e];
  }
  __syncthreads();
  double acc[4][4] = {};
  gemm_nt_64(p, q, acc, ty, tx);
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c)
      Ak[(int64_t)(ib * B + ty * 4 + r) * nf + jb * B + tx * 4 + c] = acc[r][c];
}

// Trailing update: A[ib][cb] -= L[ib][jb] * L[cb][jb]^T for jb < cb <= ib.
__global__ __launch_bounds__(256) void k_syrk(double* __restrict__ A, int nf, int jb) {
  __shared__ double p[B][LDP];
  __shared__ double q[B][LDP];
  const int k = blockIdx.y;
  // triangular tile index -> (ib, cb) with cb <= ib, both offset by jb + 1
  const int t = blockIdx.x;
  int r = static_cast<int>((sqrt(8.0 * t + 1.0) - 1.0) * 0.5);
  while ((r + 1) * (r + 2) / 2 <= t) ++r;
  while (r * (r + 1) / 2 > t) --r;
  const int ib = jb + 1 + r;
  const int cb = jb + 1 + (t - r * (r + 1) / 2);
  const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
  double* Ak = A + (int64_t)k * nf * nf;
  for (int e = tid; e < B * B; e += 256) {
    const int i = e / B, c = e % B;
    p[i][c] = Ak[(int64_t)(ib * B + i) * nf + jb * B + c];
    q[i][c] = Ak[(int64_t)(cb * B + i) * nf + jb * B + c];
  }
  __syncthreads();
  double acc[4][4] = {};
  gemm_nt_64(p, q, acc, ty, tx);
#pragma unroll
  for (int rr = 0; rr < 4; ++rr)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      double* dst = Ak + (int64_t)(ib * B + ty * 4 + rr) * nf + cb * B + tx * 4 + c;
      *dst -= acc[rr][c];
    }
}

// Inverse of the factor, one workgroup per (block column j, objective).
__global__ __launch_bounds__(256) void k_trtri(const double* __restrict__ A,
                                               const double* __restrict__ Dinv,
                                               double* __restrict__ W, int nf) {
  __shared__ double p[B][LDP];
  __shared__ double q[B][LDP];
  const int k = blockIdx.y;
  const int j = blockIdx.x;
  const int nbk = nf / B;
  const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
  const double* Ak = A + (int64_t)k * nf * nf;
  const double* Dk = Dinv + (int64_t)k * nbk * B * B;
  double* Wk = W + (int64_t)k * nf * nf;
  // W_jj = D_j^{-1}
  for (int e = tid; e < B * B; e += 256) {
    const int i = e / B, c = e % B;
    Wk[(int64_t)(j * B + i) * nf + j * B + c] = Dk[(int64_t)j * B * B + e];
  }
  __threadfence();
  __syncthreads();
  for (int i = j + 1; i < nbk; ++i) {
    // acc = sum_{t=j}^{i-1} L_it W_tj   (computed as P * Q^T with Q = W_tj^T)
    double acc[4][4] = {};
    for (int tb = j; tb < i; ++tb) {
      for (int e = tid; e < B * B; e += 256) {
        const int r = e / B, c = e % B;
        p[r][c] = Ak[(int64_t)(i * B + r) * nf + tb * B + c];
        q[c][r] = Wk[(int64_t)(tb * B + r) * nf + j * B + c];   // q = W_tj^T
      }
      __syncthreads();
      gemm_nt_64(p, q, acc, ty, tx);
      __syncthreads();
    }
    // W_ij = -D_i^{-1} acc: stage acc^T in q, D_i in p
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int c = 0; c < 4; ++c) q[tx * 4 + c][ty * 4 + r] = acc[r][c];
    for (int e = tid; e < B * B; e += 256) {
      const int r = e / B, c = e % B;
      p[r][c] = Dk[(int64_t)i * B * B + e];
    }
    __syncthreads();
    double out[4][4] = {};
    gemm_nt_64(p, q, out, ty, tx);
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        Wk[(int64_t)(i * B + ty * 4 + r) * nf + j * B + tx * 4 + c] = -out[r][c];
    __threadfence();
    __syncthreads();
  }
}

// tmp_k = W_k y_k  (one wave per row, lanes over columns)
__global__ __launch_bounds__(256) void k_wy(const double* __restrict__ W,
                                            const float* __restrict__ Y, int64_t n,
                                            int m, int nf, double* __restrict__ tmp) {
  const int k = blockIdx.y;
  const int row = blockIdx.x * 4 + threadIdx.x / 64;
  const int lane = threadIdx.x % 64;
  if (row >= nf) return;
  const double* Wr = W + ((int64_t)k * nf + row) * nf;
  double acc = 0.0;
  for (int j = lane; j <= row && j < n; j += 64)
    acc += Wr[j] * static_cast<double>(Y[(int64_t)j * m + k]);
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) tmp[(int64_t)k * nf + row] = (row < n) ? acc : 0.0;
}

// alpha_k[j] = sum_{i >= j} W_k[i][j] tmp_k[i]  (thread per column)
__global__ __launch_bounds__(256) void k_wty(const double* __restrict__ W,
                                             const double* __restrict__ tmp,
                                             int64_t n, int nf, int n_pad,
                                             float* __restrict__ alpha) {
  const int k = blockIdx.y;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= n_pad) return;
  double acc = 0.0;
  if (j < n) {
    const double* Wk = W + (int64_t)k * nf * nf;
    for (int64_t i = j; i < n; ++i) acc += Wk[i * nf + j] * tmp[(int64_t)k * nf + i];
  }
  alpha[(int64_t)k * n_pad + j] = static_cast<float>(acc);
}

// Pack lower 16x16 blocks of W into MFMA A-fragment order:
// Lp[k][blk(I,J)][lane][kk] = W[I*16 + lane%16][J*16 + 4*kk + lane/16].
__global__ __launch_bounds__(256) void k_pack(const double* __restrict__ W, int64_t n,
                                              int nf, int nb, float* __restrict__ Lp) {
  const int k = blockIdx.y;
  const int64_t nblk = (int64_t)nb * (nb + 1) / 2;
  const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;   // (blk, lane)
  if (g >= nblk * 64) return;
  const int64_t blk = g / 64;
  const int lane = static_cast<int>(g % 64);
  int I = static_cast<int>((sqrt(8.0 * blk + 1.0) - 1.0) * 0.5);
  while ((int64_t)(I + 1) * (I + 2) / 2 <= blk) ++I;
  while ((int64_t)I * (I + 1) / 2 > blk) --I;
  const int J = static_cast<int>(blk - (int64_t)I * (I + 1) / 2);
  const int row = I * kBlk + lane % 16;
  const double* Wk = W + (int64_t)k * nf * nf;
  float4 v;
  float* vp = reinterpret_cast<float*>(&v);
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    const int col = J * kBlk + 4 * kk + lane / 16;
    vp[kk] = (row < n && col < n) ? static_cast<float>(Wk[(int64_t)row * nf + col]) : 0.f;
  }
  reinterpret_cast<float4*>(Lp)[(int64_t)k * nblk * 64 + g] = v;
}

// Xs[k][i][t] = X[i][t] * invls[k][t] (zero padding beyond n and d)
__global__ __launch_bounds__(256) void k_scale_x(const float* __restrict__ X, int64_t n,
                                                 int d, int dx, int n_pad,
                                                 const float* __restrict__ invls,
                                                 float* __restrict__ Xs) {
  const int k = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)n_pad * dx) return;
  const int64_t i = e / dx;
  const int t = static_cast<int>(e % dx);
  float v = 0.f;
  if (i < n && t < d) v = X[i * d + t] * invls[k * dx + t];
  Xs[(int64_t)k * n_pad * dx + e] = v;
}

__global__ void k_lower_to_f32(const double* __restrict__ A, int64_t n, int nf,
                               float* __restrict__ L) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= n * n) return;
  const int64_t i = e / n, j = e % n;
  L[e] = (j <= i) ? static_cast<float>(A[i * nf + j]) : 0.f;
}

__global__ void k_f32_to_padded(const float* __restrict__ Asrc, int64_t n, int nf,
                                double* __restrict__ P) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)nf * nf) return;
  const int64_t i = e / nf, j = e % nf;
  double v;
  if (i < n && j < n) v = static_cast<double>(Asrc[i * n + j]);
  else v = (i == j) ? 1.0 : 0.0;
  P[e] = v;
}

}  // namespace

hipError_t launch_gram(const float* X, int64_t n, int d, int m, int n_fit,
                       const double* ls, const double* os, const double* noise,
                       double* A, hipStream_t st) {
  dim3 grid((n_fit + 15) / 16, (n_fit + 15) / 16, m), block(16, 16);
  hipLaunchKernelGGL(k_gram, grid, block, 0, st, X, n, d, n_fit, ls, os, noise, A);
  return hipGetLastError();
}

hipError_t launch_cholesky(double* A, double* Dinv, int nf, int m, int* flag,
                           hipStream_t st) {
  const int nbk = nf / B;
  for (int jb = 0; jb < nbk; ++jb) {
    hipLaunchKernelGGL(k_potrf, dim3(m), dim3(256), 0, st, A, Dinv, nf, jb, flag);
    const int T = nbk - jb - 1;
    if (T > 0) {
      hipLaunchKernelGGL(k_trsm, dim3(T, m), dim3(256), 0, st, A, Dinv, nf, jb);
      hipLaunchKernelGGL(k_syrk, dim3(T * (T + 1) / 2, m), dim3(256), 0, st, A, nf, jb);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_trtri(const double* A, const double* Dinv, double* W, int nf, int m,
                        hipStream_t st) {
  hipError_t e = hipMemsetAsync(W, 0, sizeof(double) * (size_t)m * nf * nf, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_trtri, dim3(nf / B, m), dim3(256), 0, st, A, Dinv, W, nf);
  return hipGetLastError();
}

hipError_t launch_alpha(const double* W, const float* Y, int64_t n, int m, int nf,
                        int n_pad, double* tmp, float* alpha, hipStream_t st) {
  hipLaunchKernelGGL(k_wy, dim3((nf + 3) / 4, m), dim3(256), 0, st, W, Y, n, m, nf, tmp);
  hipLaunchKernelGGL(k_wty, dim3((n_pad + 255) / 256, m), dim3(256), 0, st, W, tmp, n,
                     nf, n_pad, alpha);
  return hipGetLastError();
}

hipError_t launch_pack(const double* W, int64_t n, int m, int nf, int nb, float* Lp,
                       const float* X, int d, int dx, const float* invls, float* Xs,
                       hipStream_t st) {
  const int64_t nblk = (int64_t)nb * (nb + 1) / 2;
  const unsigned gx = static_cast<unsigned>((nblk * 64 + 255) / 256);
  hipLaunchKernelGGL(k_pack, dim3(gx, m), dim3(256), 0, st, W, n, nf, nb, Lp);
  const int n_pad = nb * kBlk;
  const unsigned gx2 = static_cast<unsigned>(((int64_t)n_pad * dx + 255) / 256);
  hipLaunchKernelGGL(k_scale_x, dim3(gx2, m), dim3(256), 0, st, X, n, d, dx, n_pad,
                     invls, Xs);
  return hipGetLastError();
}

hipError_t launch_lower_to_f32(const double* A, int64_t n, int nf, float* L,
                               hipStream_t st) {
  const unsigned g = static_cast<unsigned>((n * n + 255) / 256);
  hipLaunchKernelGGL(k_lower_to_f32, dim3(g), dim3(256), 0, st, A, n, nf, L);
  return hipGetLastError();
}

hipError_t launch_f32_to_padded(const float* A, int64_t n, int nf, double* P,
                                hipStream_t st) {
  const unsigned g = static_cast<unsigned>(((int64_t)nf * nf + 255) / 256);
  hipLaunchKernelGGL(k_f32_to_padded, dim3(g), dim3(256), 0, st, A, n, nf, P);
  return hipGetLastError();
}

}  // namespace bo
