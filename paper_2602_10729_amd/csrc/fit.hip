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
// Blocked right-looking Cholesky with 64x64 blocks that carries the inverse
// along. R starts as the identity; after step kb the block rows <= kb of W
// hold L^{-1} and the rows below hold R_i = delta_i - sum_{k<=kb} L_ik W_k
// (W itself is never cleared: each block is written before it is read).
// Every diagonal block is factored and inverted in one workgroup
// (D_kk = L_kk^{-1} lands in W's diagonal block). Step kb:
//   panel:  L_ik = A_ik D_kk^T for the rows below, W_kj = D_kk R_kj for the
//           columns left of the diagonal (quarter tiles);
//   update: trailing A_ic -= L_ik L_ck^T (kb < c <= i) and R_ij -= L_ik W_kj
//           (i > kb, j <= kb), 64x64x64 tiles on the fp64 matrix cores; the
//           workgroup that updates the next diagonal tile factors and
//           inverts it at once, so no separate factor launch is needed after
//           the first.
// Two launches per block column; the serial chain is one 64-step fused
// factor and inverse of the diagonal block per block column.
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

__device__ inline double matern32_d(double r2) {
  const double r = sqrt(r2);
  const double c = 1.73205080756887729353;   // sqrt(3)
  return (1.0 + c * r) * exp(-c * r);
}

// Gram matrix in fp64, lower block triangle only (tiles above the diagonal
// blocks are never read by the factorisation). One 16x16 tile per
// workgroup; the tile's 32 rows of X, the inverse lengthscales and (for the
// composite kernel) the rows' preference weights are staged in LDS first,
// so every global load is issued up front.
//   plain:     k = os M52(r)
//   composite: k = os M52(r_route) + s_dep w_i w_j M32(r_dep)
//                  + s_int M52(r_route) M32(r_dep)
__global__ __launch_bounds__(256) void k_gram(const float* __restrict__ X, int64_t n, int d,
                                              int nf, GramParams g, double* __restrict__ A,
                                              unsigned long long* __restrict__ kdiag, int bj0) {
  __shared__ float xs[2][16][BO_MAX_D + 1];
  __shared__ double il[BO_MAX_D];
  __shared__ double wrow[2][16];
  const int k = blockIdx.z;
  const int bi = blockIdx.y, bj = bj0 + blockIdx.x;   // 16x16 tiles from tile column bj0
  if ((bj >> 2) > (bi >> 2)) return;                // strictly above the 64-block diagonal
  const int tid = threadIdx.y * 16 + threadIdx.x;
  // rows bi*16.. (s = 0) and bj*16.. (s = 1); rows past n read as 0
  for (int e = tid; e < 32 * d; e += 256) {
    const int s = e / (16 * d), rem = e % (16 * d), r = rem / d, t = rem % d;
    const int64_t row = (int64_t)(s ? bj : bi) * 16 + r;
    xs[s][r][t] = (row < n) ? X[row * d + t] : 0.f;
  }
  if (tid < d) il[tid] = g.ils[k * d + tid];
  __syncthreads();
  const int dr = g.dr;
  if (dr > 0 && tid < 32) {
    const int s = tid >> 4, r = tid & 15;
    const double* p = g.pref + (int64_t)k * (d - dr);
    double e = 0.0;
    for (int t = dr; t < d; ++t) e = fma(p[t - dr], static_cast<double>(xs[s][r][t]), e);
    wrow[s][r] = exp(e);
  }
  __syncthreads();
  const int i = bi * 16 + threadIdx.y;
  const int j = bj * 16 + threadIdx.x;
  if (i >= nf || j >= nf) return;
  double v;
  if (i < n && j < n) {
    double ra = 0.0, rb = 0.0;          // routing / deployment (plain: all in ra)
    for (int t = 0; t < d; ++t) {
      const double diff = (static_cast<double>(xs[0][threadIdx.y][t]) -
                           static_cast<double>(xs[1][threadIdx.x][t])) * il[t];
      if (dr > 0 && t >= dr) rb = fma(diff, diff, rb);
      else ra = fma(diff, diff, ra);
    }
    if (dr == 0) {
      v = matern52_d(ra, g.os[k]);
    } else {
      const double k5 = matern52_d(ra, 1.0), k3 = matern32_d(rb);
      v = g.os[k] * k5 + g.s_dep[k] * wrow[0][threadIdx.y] * wrow[1][threadIdx.x] * k3 +
          g.s_int[k] * k5 * k3;
    }
    if (i == j) {
      v += g.noise[k];
      // largest diagonal entry per objective (non-negative doubles order
      // like their bit patterns)
      if (kdiag) atomicMax(kdiag + k, static_cast<unsigned long long>(__double_as_longlong(v)));
    }
  } else {
    v = (i == j) ? 1.0 : 0.0;
  }
  A[((int64_t)k * nf + i) * nf + j] = v;
}

// Composite: fp32 preference weights of the training points for scoring.
__global__ __launch_bounds__(256) void k_weights(const float* __restrict__ X, int64_t n, int d,
                                                 int n_pad, GramParams g,
                                                 float* __restrict__ wts) {
  const int k = blockIdx.y;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_pad) return;
  float w = 0.f;
  if (i < n) {
    const double* p = g.pref + (int64_t)k * (d - g.dr);
    double e = 0.0;
    for (int t = g.dr; t < d; ++t) e = fma(p[t - g.dr], static_cast<double>(X[i * d + t]), e);
    w = static_cast<float>(exp(e));
  }
  wts[(int64_t)k * n_pad + i] = w;
}

// 1 / sqrt(d), d > 0: the hardware estimate refined by two Newton steps
// y <- y (3 - d y^2) / 2, each of which roughly squares the relative error.
__device__ __forceinline__ double rsqrt_d(double d) {
  double y = __builtin_amdgcn_rsq(d);
  const double h = 0.5 * d;
  y = y * fma(-h * y, y, 1.5);
  return y * fma(-h * y, y, 1.5);
}

// Factor the symmetric 64x64 block held in LDS `a` (lower triangle read) and
// invert the factor: on return a = L (zeros above the diagonal) and
// x = L^{-1} (zeros above the diagonal). All eight waves of the 512-thread
// workgroup take part (every thread must call this), two per SIMD so that
// one wave's multiply-adds fill the other's wait on the pivot chain: thread
// (w, c) = (wave, lane) keeps, in registers indexed only by unrolled
// constants,
//   row c of A, columns 8w .. 8w+7, and
//   column c of X, rows 8w .. 8w+7.
//
// The factor (right-looking, unscaled) and the inverse (forward
// substitution, one column of X per lane) advance together, one barrier per
// step j; only the wave holding column j of A and row j of X writes:
//   before the barrier it publishes column j of A as it stands
//   (A_ij = L_ij L_jj for rows i > j, zeros for rows <= j; one write of the
//   whole wave), the pivot A_jj, and row j of X as it stands (X_jc L_jj);
//   the buffers are double-buffered by step parity;
//   after it, every thread takes 1 / L_jj = A_jj^{-1/2} and updates
//     A_ic -= A_ij A_cj / A_jj   (its row i, its 8 columns c)
//     X_ic -= A_ij (X_jc L_jj) / A_jj   (its column c, its 8 rows i);
//   the zeros of the published column leave rows and columns <= j as they
//   are (above the diagonal A is never read again; rows of X up to j are
//   final).
// Row j of X keeps the factor L_jj until the end, where every row of X and
// every column of A is scaled by its 1 / L_jj.
// A non-positive or non-finite pivot sets *flag and is replaced by 1.
// Scratch: scr holds 6 x 64 doubles, 16-byte aligned (two published columns
// of A, two published rows of X, two pivots, the 64 values 1 / L_jj).
constexpr int kFactorThreads = 512;
__device__ __forceinline__ void chol_inv64(double (*a)[LDP], double (*x)[LDP], double* scr,
                                           int* flag) {
  const int c = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // column group 8w ..
  double* colbuf = scr;                      // [2][64] column j of A, rows > j
  double* rowbuf = scr + 2 * B;              // [2][64] row j of X
  double* pivbuf = scr + 4 * B;              // [2]     A_jj
  double* rdiag = scr + 5 * B;               // [64]    1 / L_jj
  double r[8], xv[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    r[t] = a[c][8 * w + t];
    xv[t] = (8 * w + t == c) ? 1.0 : 0.0;
  }
  bool bad_any = false;
  // steps j = 8 jw + jt: the group of the pivot is a loop variable and the
  // position within it an unrolled constant (register indices stay constant
  // while the straight-line code stays one group long)
#pragma unroll 1
  for (int jw = 0; jw < 8; ++jw) {
#pragma unroll
  for (int jt = 0; jt < 8; ++jt) {
    const int j = 8 * jw + jt;
    double* col = colbuf + (jt & 1) * B;
    double* row = rowbuf + (jt & 1) * B;
    if (w == jw) {
      col[c] = (c > j) ? r[jt] : 0.0;       // A_cj of this lane's row c
      row[c] = xv[jt];                      // X_jc before its division by L_jj
      if (c == j) pivbuf[jt & 1] = r[jt];
    }
    __syncthreads();
    // every read of the step is issued together, ahead of the arithmetic
    const double a_jj = pivbuf[jt & 1];
    const double a_cj = col[c];
    const double x_jc = row[c];
    double2 l[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) l[t] = *reinterpret_cast<const double2*>(col + 8 * w + 2 * t);
    __builtin_amdgcn_sched_barrier(0);
    const bool bad = !(a_jj > 0.0) || !isfinite(a_jj);
    const double d = bad ? 1.0 : a_jj;
    bad_any = bad_any || bad;
    const double isd = rsqrt_d(d);
    const double id = isd * isd;
    const double mrow = a_cj * id;          // A_cj / A_jj for this lane's row c
    const double xs = x_jc * id;            // (X_jc / L_jj) / L_jj
#pragma unroll
    for (int t = 0; t < 8; t += 2) {
      r[t] = fma(-mrow, l[t / 2].x, r[t]);
      r[t + 1] = fma(-mrow, l[t / 2].y, r[t + 1]);
      xv[t] = fma(-l[t / 2].x, xs, xv[t]);
      xv[t + 1] = fma(-l[t / 2].y, xs, xv[t + 1]);
    }
    if (threadIdx.x == 0) rdiag[j] = isd;
  }
  }
  if (bad_any && threadIdx.x == 0) atomicOr(flag, 1);   // every thread saw every pivot
  __syncthreads();   // rdiag is complete; every published read is done
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const int k = 8 * w + t;                // column of A / row of X
    a[c][k] = (c >= k) ? r[t] * rdiag[k] : 0.0;
    x[k][c] = xv[t] * rdiag[k];
  }
  __syncthreads();
}

// Copies of 64x64 tiles between global memory (leading dimension ld) and
// padded LDS tiles, by the first 256 threads of a workgroup. Every load of a call is
// issued before the first LDS store, so the latencies overlap; two tiles
// can be fetched in one call. Transposed variants store dst[c][i] = src[i][c].
template <bool T>
__device__ __forceinline__ void put_tile(double (*dst)[LDP], const double (&v)[16]) {
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int e = threadIdx.x + 256 * k, i = e >> 6, c = e & 63;
    if (T) dst[c][i] = v[k];
    else dst[i][c] = v[k];
  }
}

__device__ __forceinline__ void get_tile(double (&v)[16], const double* src, int ld) {
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int e = threadIdx.x + 256 * k, i = e >> 6, c = e & 63;
    v[k] = src[(int64_t)i * ld + c];
  }
}

template <bool T0 = false>
__device__ inline void load_block(double (*dst)[LDP], const double* src, int ld) {
  double v[16];
  get_tile(v, src, ld);
  put_tile<T0>(dst, v);
}

template <bool T0, bool T1>
__device__ inline void load_blocks(double (*d0)[LDP], const double* s0, double (*d1)[LDP],
                                   const double* s1, int ld) {
  double v0[16], v1[16];
  get_tile(v0, s0, ld);
  get_tile(v1, s1, ld);
  put_tile<T0>(d0, v0);
  put_tile<T1>(d1, v1);
}

__device__ inline void store_block(double* dst, int ld, const double (*srcb)[LDP]) {
  for (int e = threadIdx.x; e < B * B; e += blockDim.x) {
    const int i = e >> 6, c = e & 63;
    dst[(int64_t)i * ld + c] = srcb[i][c];
  }
}

// First diagonal block (kb = 0) of every objective: L into A, L^{-1} into W.
// Eight waves (the factor's layout); the first four load the tile.
__global__ __launch_bounds__(kFactorThreads) void k_factor_first(double* __restrict__ A,
                                                                 double* __restrict__ W, int nf,
                                                                 int* __restrict__ flag) {
  __shared__ double a[B][LDP];
  __shared__ __align__(16) double x[B][LDP];
  __shared__ __align__(16) double scr[6 * B];
  double* Ak = A + (int64_t)blockIdx.x * nf * nf;
  double* Wk = W + (int64_t)blockIdx.x * nf * nf;
  if (threadIdx.x < 256) load_block(a, Ak, nf);
  __syncthreads();
  chol_inv64(a, x, scr, flag);
  store_block(Ak, nf, a);
  store_block(Wk, nf, x);
}

typedef double doublex4 __attribute__((ext_vector_type(4)));

// 64x64x64 product on the fp64 matrix cores (v_mfma_f64_16x16x4f64: A[i][k]
// from lane i + 16k, B[k][j] from lane j + 16k, D[i][j] in lane
// j + 16(i%4), element i/4): wave w (of the first four) adds
// sum_t P[i][t] Q[c][t] over its 32x32 quadrant, rows 32(w/2).., columns
// 32(w%2).., as 2x2 tiles of 16x16;
// acc[a][b][v] is element (32(w/2) + 16a + lane/16 + 4v,
// 32(w%2) + 16b + lane%16) (tile_row / tile_col below).
__device__ __forceinline__ void gemm_nt_64(const double (*P)[LDP], const double (*Q)[LDP],
                                           doublex4 (&acc)[2][2]) {
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r0 = 32 * (w >> 1) + (l & 15), c0 = 32 * (w & 1) + (l & 15), kq = l >> 4;
#pragma unroll 4
  for (int t = 0; t < B; t += 4) {
    const double a0 = P[r0][t + kq], a1 = P[r0 + 16][t + kq];
    const double b0 = Q[c0][t + kq], b1 = Q[c0 + 16][t + kq];
    acc[0][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, acc[0][0], 0, 0, 0);
    acc[0][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, acc[0][1], 0, 0, 0);
    acc[1][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, acc[1][0], 0, 0, 0);
    acc[1][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, acc[1][1], 0, 0, 0);
  }
}
__device__ __forceinline__ int tile_row(int a, int v) {
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  return 32 * (w >> 1) + 16 * a + (l >> 4) + 4 * v;
}
__device__ __forceinline__ int tile_col(int b) {
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  return 32 * (w & 1) + 16 * b + (l & 15);
}

// Panel of step kb, with D = L_kk^{-1} (held in W's diagonal block kb), in
// quarters (u = blockIdx.x % 4) so that its T + kb tiles fill four times as
// many workgroups:
// tiles t < T: A[kb+1+t][kb] <- A[kb+1+t][kb] D^T (rows below the diagonal);
//   quarter u takes rows 16u .. 16u+15 of the tile, the only rows it reads;
// tiles T <= t < T + kb: W[kb][jb] <- D R[kb][jb] for jb = t - T (< kb);
//   quarter u takes columns 16u .. 16u+15 of R, the only columns it reads.
// The products run on the fp64 matrix cores, each wave one 16x16 tile.
__global__ __launch_bounds__(256) void k_panel(double* __restrict__ A, double* __restrict__ W,
                                               int nf, int kb) {
  __shared__ double p[B][LDP];
  __shared__ double q[B][LDP];
  const int k = blockIdx.y;
  const int nbk = nf / B;
  const int T = nbk - kb - 1;
  const int t = blockIdx.x >> 2, u = blockIdx.x & 3;
  const int tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  double* Ak = A + (int64_t)k * nf * nf;
  double* Wk = W + (int64_t)k * nf * nf;
  const int o = kb * B;
  const double* D = Wk + (int64_t)o * nf + o;
  double v0[4], v1[16];
  if (t < T) {
    double* dst = Ak + (int64_t)(kb + 1 + t) * B * nf + o + (int64_t)16 * u * nf;
    // p[i][s] = tile row 16u + i (i < 16), q[c][s] = D[c][s]
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int g = tid + 256 * e;
      v0[e] = dst[(int64_t)(g >> 6) * nf + (g & 63)];
    }
    get_tile(v1, D, nf);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int g = tid + 256 * e;
      p[g >> 6][g & 63] = v0[e];
    }
    put_tile<false>(q, v1);
    __syncthreads();
    // wave w: output columns 16w .. 16w+15 (one 16x16 tile on the matrix cores)
    doublex4 acc = {};
#pragma unroll 4
    for (int s2 = 0; s2 < B; s2 += 4)
      acc = __builtin_amdgcn_mfma_f64_16x16x4f64(p[l & 15][s2 + (l >> 4)],
                                                 q[16 * w + (l & 15)][s2 + (l >> 4)], acc, 0, 0,
                                                 0);
#pragma unroll
    for (int v = 0; v < 4; ++v)
      dst[(int64_t)((l >> 4) + 4 * v) * nf + 16 * w + (l & 15)] = acc[v];
  } else {
    double* dst = Wk + (int64_t)o * nf + (t - T) * B + 16 * u;
    // p = D; q[c][s] = R[s][16u + c] (c < 16)
    get_tile(v1, D, nf);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int g = tid + 256 * e;
      v0[e] = dst[(int64_t)(g >> 4) * nf + (g & 15)];
    }
    put_tile<false>(p, v1);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int g = tid + 256 * e;
      q[g & 15][g >> 4] = v0[e];
    }
    __syncthreads();
    // wave w: output rows 16w .. 16w+15
    doublex4 acc = {};
#pragma unroll 4
    for (int s2 = 0; s2 < B; s2 += 4)
      acc = __builtin_amdgcn_mfma_f64_16x16x4f64(p[16 * w + (l & 15)][s2 + (l >> 4)],
                                                 q[l & 15][s2 + (l >> 4)], acc, 0, 0, 0);
#pragma unroll
    for (int v = 0; v < 4; ++v)
      dst[(int64_t)(16 * w + (l >> 4) + 4 * v) * nf + (l & 15)] = acc[v];
  }
}

// Update of step kb. Tile t < T(T+1)/2: trailing A tile; the rest: R tiles
// of W (the tiles of block column kb are written, not updated: nothing
// before this step writes them). Tile 0 is the next diagonal block,
// factored and inverted right after its update (L into A, L^{-1} into W's
// diagonal block kb+1).
__global__ __launch_bounds__(kFactorThreads) void k_update(double* __restrict__ A,
                                                           double* __restrict__ W, int nf,
                                                           int kb, int* __restrict__ flag) {
  __shared__ double p[B][LDP];
  __shared__ __align__(16) double q[B][LDP];
  __shared__ __align__(16) double scr[6 * B];
  const int k = blockIdx.y;
  const int nbk = nf / B;
  const int T = nbk - kb - 1;
  const int nsyrk = T * (T + 1) / 2;
  const int t = blockIdx.x;
  double* Ak = A + (int64_t)k * nf * nf;
  double* Wk = W + (int64_t)k * nf * nf;
  const int o = kb * B;
  // eight waves (the diagonal factor's layout): the first four load and
  // multiply the tile, all eight factor the next diagonal block
  const bool prod = threadIdx.x < 256;
  double* dst;
  bool first_r = false;
  if (t < nsyrk) {
    // (ib, cb) with kb < cb <= ib: tile index t -> row r, column within row
    int r = static_cast<int>((sqrt(8.0 * t + 1.0) - 1.0) * 0.5);
    while ((r + 1) * (r + 2) / 2 <= t) ++r;
    while (r * (r + 1) / 2 > t) --r;
    const int ib = kb + 1 + r;
    const int cb = kb + 1 + (t - r * (r + 1) / 2);
    if (prod)
      load_blocks<false, false>(p, Ak + (int64_t)ib * B * nf + o,      // L[ib][kb]
                                q, Ak + (int64_t)cb * B * nf + o, nf); // L[cb][kb]
    dst = Ak + (int64_t)ib * B * nf + cb * B;
  } else {
    // R tile (ib, jb): ib > kb, jb <= kb:  W[ib][jb] -= L[ib][kb] W[kb][jb]
    const int u = t - nsyrk;
    const int ib = kb + 1 + u / (kb + 1);
    const int jb = u % (kb + 1);
    first_r = (jb == kb);
    if (prod)
      load_blocks<false, true>(p, Ak + (int64_t)ib * B * nf + o,        // L[ib][kb]
                               q, Wk + (int64_t)o * nf + jb * B, nf);   // q = W[kb][jb]^T
    dst = Wk + (int64_t)ib * B * nf + jb * B;
  }
  // the tile's current values, requested before the product: the first
  // update of an R tile (jb = kb) starts from zero instead (W is not cleared
  // beforehand; its blocks above the diagonal are never read)
  doublex4 cur[2][2] = {};
  if (prod) {
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          cur[a][b][v] = first_r ? 0.0 : dst[(int64_t)tile_row(a, v) * nf + tile_col(b)];
  }
  __syncthreads();
  doublex4 acc[2][2] = {};
  if (prod) {
    gemm_nt_64(p, q, acc);
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        acc[a][b] = cur[a][b] - acc[a][b];
        // the next diagonal tile (t = 0) is stored once, factored, below
        if (t != 0)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            dst[(int64_t)tile_row(a, v) * nf + tile_col(b)] = acc[a][b][v];
      }
  }
  if (t == 0) {
    // next diagonal block: stage the updated tile, factor and invert it
    __syncthreads();
    if (prod) {
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int v = 0; v < 4; ++v) p[tile_row(a, v)][tile_col(b)] = acc[a][b][v];
    }
    __syncthreads();
    chol_inv64(p, q, scr, flag);
    const int o1 = o + B;
    store_block(dst, nf, p);
    store_block(Wk + (int64_t)o1 * nf + o1, nf, q);
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

// alpha_k[j] = sum_{i >= j} W_k[i][j] tmp_k[i]: 16 columns per block, 16 row
// phases per column with two accumulators each (several loads in flight),
// combined in LDS.
__global__ __launch_bounds__(256) void k_wty(const double* __restrict__ W,
                                             const double* __restrict__ tmp,
                                             int64_t n, int nf, int n_pad,
                                             float* __restrict__ alpha,
                                             double* __restrict__ alpha64) {
  __shared__ double part[16][17];
  const int k = blockIdx.y;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int j = blockIdx.x * 16 + tx;
  double a0 = 0.0, a1 = 0.0;
  if (j < n) {
    const double* Wk = W + (int64_t)k * nf * nf;
    const double* tk = tmp + (int64_t)k * nf;
    int64_t i = j + ty;
    for (; i + 16 < n; i += 32) {
      a0 = fma(Wk[i * nf + j], tk[i], a0);
      a1 = fma(Wk[(i + 16) * nf + j], tk[i + 16], a1);
    }
    if (i < n) a0 = fma(Wk[i * nf + j], tk[i], a0);
  }
  part[ty][tx] = a0 + a1;
  __syncthreads();
  if (ty == 0 && j < n_pad) {
    double v = 0.0;
#pragma unroll
    for (int t = 0; t < 16; ++t) v += part[t][tx];
    alpha[(int64_t)k * n_pad + j] = (j < n) ? static_cast<float>(v) : 0.f;
    if (alpha64 && j < nf) alpha64[(int64_t)k * nf + j] = (j < n) ? v : 0.0;
  }
}

// Power-of-two scale of each 16-row block of W = L^{-1} for its fp16 split:
// with mx the largest |W| over the block's lower entries, mx = f 2^E
// (f in [0.5, 1)), the pack stores W 2^(14 - E), so every entry of the block
// is at most 2^14 in magnitude (fp16 holds up to 65504) and the low halves of
// all entries above 2^-3 of that are normal fp16 numbers; rsc[k][I] = 2^(E-14)
// undoes it (stored after objective k's fragment blocks: rsc + k * stride,
// followed by a zero at entry nb for row blocks past the matrix).
// wmax[k] gets the largest |W| of objective k (bit pattern of a non-negative
// double), for the conditioning estimate; a non-finite entry sets *flag. One
// workgroup per (row block, objective).
__global__ __launch_bounds__(256) void k_rowblock_scale(const double* __restrict__ W, int64_t n,
                                                        int nf, float* __restrict__ rsc,
                                                        int64_t stride,
                                                        unsigned long long* __restrict__ wmax,
                                                        int* __restrict__ flag) {
  __shared__ double part[256];
  const int I = blockIdx.x, k = blockIdx.y;
  const double* Wk = W + (int64_t)k * nf * nf;
  // the block's 16 rows, columns 0 .. 16I + 15: consecutive threads take
  // consecutive columns (coalesced), the 16 rows in turn
  const int64_t lim = (int64_t)I * kBlk + kBlk;
  const int64_t ncol = (lim < n) ? lim : n;
  double mx = 0.0;
  bool bad = false;
  for (int64_t col = threadIdx.x; col < ncol; col += 256) {
    double v[kBlk];
#pragma unroll
    for (int r = 0; r < kBlk; ++r) {
      const int64_t row = (int64_t)I * kBlk + r;
      v[r] = (row < n && col <= row) ? Wk[row * nf + col] : 0.0;
    }
#pragma unroll
    for (int r = 0; r < kBlk; ++r) {
      bad = bad || !(fabs(v[r]) < INFINITY);
      mx = fmax(mx, fabs(v[r]));
    }
  }
  if (bad) *flag = 1;
  part[threadIdx.x] = mx;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (static_cast<int>(threadIdx.x) < h)
      part[threadIdx.x] = fmax(part[threadIdx.x], part[threadIdx.x + h]);
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double m = part[0];
    int E = 0;
    if (m > 0.0) (void)frexp(m, &E);
    rsc[(int64_t)k * stride + I] = ldexpf(1.0f, E - 14);
    if (I == 0) rsc[(int64_t)k * stride + gridDim.x] = 0.f;   // entry nb: past the matrix
    atomicMax(wmax + k, static_cast<unsigned long long>(__double_as_longlong(m)));
  }
}

// The same row-block maxima spread over column chunks: workgroup (I, c, k)
// takes columns 256c .. 256c+255 of row block I's lower entries and merges
// its largest |W| into bmax[k][I] (bit pattern of a non-negative double,
// zeroed by the caller); a non-finite entry sets *flag.
__global__ __launch_bounds__(256) void k_rowblock_max(const double* __restrict__ W, int64_t n,
                                                      int nf, int nb,
                                                      unsigned long long* __restrict__ bmax,
                                                      int* __restrict__ flag) {
  __shared__ double part[4];
  const int I = blockIdx.x, k = blockIdx.z;
  const int64_t lim = (int64_t)I * kBlk + kBlk;
  const int64_t ncol = (lim < n) ? lim : n;
  const int64_t col = (int64_t)blockIdx.y * 256 + threadIdx.x;
  if ((int64_t)blockIdx.y * 256 >= ncol) return;          // the whole workgroup
  const double* Wk = W + (int64_t)k * nf * nf;
  double mx = 0.0;
  bool bad = false;
  if (col < ncol) {
    double v[kBlk];
#pragma unroll
    for (int r = 0; r < kBlk; ++r) {
      const int64_t row = (int64_t)I * kBlk + r;
      v[r] = (row < n && col <= row) ? Wk[row * nf + col] : 0.0;
    }
#pragma unroll
    for (int r = 0; r < kBlk; ++r) {
      bad = bad || !(fabs(v[r]) < INFINITY);
      mx = fmax(mx, fabs(v[r]));
    }
  }
  if (bad) *flag = 1;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o));
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = mx;
  __syncthreads();
  if (threadIdx.x == 0) {
    const double m = fmax(fmax(part[0], part[1]), fmax(part[2], part[3]));
    atomicMax(bmax + (int64_t)k * nb + I, static_cast<unsigned long long>(__double_as_longlong(m)));
  }
}

// Pack the lower triangle of W = L^{-1} as fp16 hi/lo MFMA A fragments of
// 16-row x 32-column blocks (the scoring path's operand format):
// row block I holds the blocks J = 0 .. I/2, block (I, J) at index
// start(I) + J with start(2t) = t(t+1), start(2t+1) = (t+1)^2, followed by one
// zero block (index start(nb), which maps to rows >= n). Each block is 2 KiB:
// the hi plane, then the lo plane, 16 bytes per lane, lane l element e being
// W[16I + l%16][32J + 8(l/16) + e] (zero above the diagonal and past n),
// scaled by its row block's power of two (w = W / rsc[I], exact) and split as
// hi = fp16(w), lo = fp16(w - hi).
__global__ __launch_bounds__(256) void k_pack(const double* __restrict__ W, int64_t n,
                                              int nf, int64_t nblk, int nb,
                                              float* __restrict__ rsc, int64_t stride,
                                              _Float16* __restrict__ Lp,
                                              const unsigned long long* __restrict__ bmax,
                                              unsigned long long* __restrict__ wmax) {
  const int k = blockIdx.y;
  const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;   // (blk, lane)
  if (g >= nblk * 64) return;
  const int64_t blk = g / 64;
  const int lane = static_cast<int>(g % 64);
  // row block I of blk: start(I) <= blk < start(I + 1)
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
  const int64_t row = (int64_t)I * kBlk + lane % 16;
  const double* Wk = W + (int64_t)k * nf * nf;
  // the zero block (I = nb) has no scale; with bmax the scale of row block I
  // is taken here from its maximum (the first block of the row stores it)
  float rs = 1.0f;
  if (I < nb) {
    if (bmax) {
      const double mI = __longlong_as_double(static_cast<long long>(bmax[(int64_t)k * nb + I]));
      int E = 0;
      if (mI > 0.0) (void)frexp(mI, &E);
      rs = ldexpf(1.0f, E - 14);
      if (J == 0 && lane == 0) {
        rsc[(int64_t)k * stride + I] = rs;
        atomicMax(wmax + k, static_cast<unsigned long long>(__double_as_longlong(mI)));
      }
    } else {
      rs = rsc[(int64_t)k * stride + I];
    }
  } else if (bmax && lane == 0) {
    rsc[(int64_t)k * stride + nb] = 0.f;      // entry nb: past the matrix
  }
  const double sc = (I < nb) ? 1.0 / static_cast<double>(rs) : 1.0;
  _Float16 hi[8], lo[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int64_t col = (int64_t)J * 32 + 8 * (lane / 16) + e;
    const double w = (row < n && col < n && col <= row) ? Wk[row * nf + col] * sc : 0.0;
    const _Float16 h = static_cast<_Float16>(static_cast<float>(w));
    hi[e] = h;
    lo[e] = static_cast<_Float16>(static_cast<float>(w - static_cast<double>(h)));
  }
  _Float16* dst = Lp + (int64_t)k * 2 * stride + blk * 1024 + lane * 8;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    dst[e] = hi[e];
    dst[512 + e] = lo[e];
  }
}

// Xs[k][i][t] = X[i][slot_dim(t)] * invls[k][t] (zero for padding slots and
// rows beyond n), with invls[k][t] = fp32(ils[k][slot_dim(t)]) also written
// out (the fp64 inverse lengthscale rounded to fp32 is the fp32 quotient
// 1 / lengthscale: double rounding is exact for a quotient when the wider
// format has at least 2p + 2 bits). Objective 0 also copies X into Xd;
// (composite) fp32 preference slopes come from their fp64 copies, and (fp64
// scoring) ils is copied into ils64.
__global__ __launch_bounds__(256) void k_scale_x(const float* __restrict__ X, int64_t n,
                                                 int d, int dx, int dr, int dr4, int n_pad,
                                                 const double* __restrict__ ils,
                                                 float* __restrict__ invls,
                                                 const double* __restrict__ pref_d,
                                                 float* __restrict__ pref, int dc,
                                                 float* __restrict__ Xd,
                                                 double* __restrict__ ils64,
                                                 float* __restrict__ Xs) {
  const int k = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)n_pad * dx) return;
  const int64_t i = e / dx;
  const int t = static_cast<int>(e % dx);
  const int c = slot_dim(t, d, dr, dr4);
  const float il = (c >= 0) ? static_cast<float>(ils[k * d + c]) : 0.f;
  float v = 0.f;
  if (i < n && c >= 0) v = X[i * d + c] * il;
  Xs[(int64_t)k * n_pad * dx + e] = v;
  if (i == 0) invls[k * dx + t] = il;
  if (k == 0 && e < n * d) Xd[e] = X[e];
  if (pref && e < dc) pref[k * dc + e] = static_cast<float>(pref_d[k * dc + e]);
  if (ils64 && e < d) ils64[k * d + e] = ils[k * d + e];
}

// ctr[k][t] = mean over the n rows of Xs[k][i][t] (fp64 sum, fp32 result):
// one block per (coordinate t, objective k), rows strided over the threads,
// then a tree sum in LDS
__global__ __launch_bounds__(256) void k_center_x(const float* __restrict__ Xs, int64_t n,
                                                  int n_pad, int dx, float* __restrict__ ctr) {
  __shared__ double part[256];
  const int t = blockIdx.x, k = blockIdx.y;
  const float* x = Xs + (int64_t)k * n_pad * dx + t;
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 256) acc += x[i * dx];
  part[threadIdx.x] = acc;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (static_cast<int>(threadIdx.x) < h) part[threadIdx.x] += part[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) ctr[k * dx + t] = static_cast<float>(part[0] / static_cast<double>(n));
}

// One thread per (row group g, fragment f, lane l): the eight fp16 values of
// the A fragment of v_mfma_f32_16x16x32_f16 that lane l supplies (row 16g +
// l%16, positions 8(l/16) .. +7 of the fragment's 32), from the centred row
// xc = Xs - ctr: stream 0 holds hi(xc[p]) at p < dx, stream 1 lo(xc[p]) at
// p < dx and hi(xc[p - dx]) at dx <= p < 2dx; zero elsewhere and for rows
// past n.
__global__ __launch_bounds__(256) void k_pack_x(const float* __restrict__ Xs, int64_t n,
                                                int n_pad, int nb, int dx,
                                                const float* __restrict__ ctr,
                                                _Float16* __restrict__ xf) {
  const int k = blockIdx.y;
  const int nf = dist_frags(dx), f0 = dist_frags0(dx);
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)nb * nf * 64) return;
  const int l = static_cast<int>(idx % 64);
  const int f = static_cast<int>((idx / 64) % nf);
  const int64_t g = idx / (64 * nf);
  const int64_t i = 16 * g + (l & 15);
  const float* x = Xs + ((int64_t)k * n_pad + i) * dx;
  const float* c = ctr + k * dx;
  _Float16* dst = xf + (((int64_t)k * nb + g) * nf + f) * 512 + l * 8;
  for (int e = 0; e < 8; ++e) {
    const int p = 32 * (f < f0 ? f : f - f0) + 8 * (l >> 4) + e;
    _Float16 v = static_cast<_Float16>(0.0f);
    if (i < n) {
      if (f < f0) {
        if (p < dx) v = static_cast<_Float16>(x[p] - c[p]);
      } else if (p < dx) {
        const float xc = x[p] - c[p];
        const _Float16 h = static_cast<_Float16>(xc);
        v = static_cast<_Float16>((xc - static_cast<float>(h)) * kDistLoScale);
      } else if (p < 2 * dx) {
        v = static_cast<_Float16>(x[p - dx] - c[p - dx]);
      }
    }
    dst[e] = v;
  }
}

// x2[k][0][i] = sum over routing slots (t < 4*dr4) of (Xs - ctr)^2, x2[k][1][i]
// over the others, both fp32 in slot order; zero for rows past n
__global__ __launch_bounds__(256) void k_norm_x(const float* __restrict__ Xs, int64_t n,
                                                int n_pad, int dx, int dr4,
                                                const float* __restrict__ ctr,
                                                float* __restrict__ x2) {
  const int k = blockIdx.y;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_pad) return;
  float g0 = 0.f, g1 = 0.f;
  if (i < n) {
    const float* x = Xs + ((int64_t)k * n_pad + i) * dx;
    const float* c = ctr + k * dx;
    for (int t = 0; t < dx; ++t) {
      const float v = x[t] - c[t];
      if (t < 4 * dr4) g0 = fmaf(v, v, g0);
      else g1 = fmaf(v, v, g1);
    }
  }
  x2[((int64_t)k * 2 + 0) * n_pad + i] = g0;
  x2[((int64_t)k * 2 + 1) * n_pad + i] = g1;
}

// ---- log marginal likelihood and its gradient ------------------------------
//
// value = -1/2 y^T K^{-1} y - sum_i log L_ii - n/2 log(2 pi), with
// y^T K^{-1} y = |W y|^2 (tmp = W y); gradient over theta = (log l, log s,
// log eta): 1/2 sum_{i,i'} (alpha_i alpha_i' - Kinv_ii') dK_ii'/dtheta.

// out[k][0] = value (one workgroup per objective)
__global__ __launch_bounds__(256) void k_logdet_quad(const double* __restrict__ A,
                                                     const double* __restrict__ tmp,
                                                     int64_t n, int nf, double* __restrict__ out,
                                                     int d) {
  __shared__ double red[2][4];
  const int k = blockIdx.x;
  const double* Ak = A + (int64_t)k * nf * nf;
  const double* tk = tmp + (int64_t)k * nf;
  double q = 0.0, ld = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 256) {
    q = fma(tk[i], tk[i], q);
    ld += log(Ak[i * nf + i]);
  }
  for (int off = 32; off > 0; off >>= 1) {
    q += __shfl_xor(q, off);
    ld += __shfl_xor(ld, off);
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[0][w] = q;
    red[1][w] = ld;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const double qq = red[0][0] + red[0][1] + red[0][2] + red[0][3];
    const double ll = red[1][0] + red[1][1] + red[1][2] + red[1][3];
    out[(int64_t)k * (d + 3)] =
        -0.5 * qq - ll - 0.5 * static_cast<double>(n) * 1.83787706640934548356;   // log(2 pi)
  }
}

// K^{-1} = W^T W into the lower 64-blocks of A: tile (I, J), I >= J, sums
// W[K][I]^T W[K][J] over K >= I (W is zero above its diagonal).
__global__ __launch_bounds__(256) void k_kinv(double* __restrict__ A, const double* __restrict__ W,
                                              int nf) {
  __shared__ double p[B][LDP];
  __shared__ double q[B][LDP];
  const int k = blockIdx.y;
  const int t = blockIdx.x;
  int I = static_cast<int>((sqrt(8.0 * t + 1.0) - 1.0) * 0.5);
  while ((I + 1) * (I + 2) / 2 <= t) ++I;
  while (I * (I + 1) / 2 > t) --I;
  const int J = t - I * (I + 1) / 2;
  const int nbk = nf / B;
  const double* Wk = W + (int64_t)k * nf * nf;
  doublex4 acc[2][2] = {};
  for (int K = I; K < nbk; ++K) {
    __syncthreads();   // the previous step's tiles are no longer read
    load_blocks<true, true>(p, Wk + (int64_t)K * B * nf + I * B,
                            q, Wk + (int64_t)K * B * nf + J * B, nf);
    __syncthreads();
    gemm_nt_64(p, q, acc);
  }
  double* dst = A + (int64_t)k * nf * nf + (int64_t)I * B * nf + J * B;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 4; ++v) dst[(int64_t)tile_row(a, v) * nf + tile_col(b)] = acc[a][b][v];
}

// Gradient partials of one 16x16 tile of observation pairs (i >= i') per
// workgroup: [tile][d + 2] = 1/2 sum w (alpha_i alpha_i' - Kinv_ii') dK/dtheta,
// w = 2 off the diagonal (the symmetric partner), 1 on it.
__global__ __launch_bounds__(256) void k_mll_grad(const float* __restrict__ X, int64_t n, int d,
                                                  int nf, GramParams g,
                                                  const double* __restrict__ A,
                                                  const double* __restrict__ alpha64,
                                                  double* __restrict__ partials) {
  __shared__ double red[4][BO_MAX_D + 2];
  const int k = blockIdx.y;
  const int64_t t = blockIdx.x;
  int64_t bi = static_cast<int64_t>((sqrt(8.0 * t + 1.0) - 1.0) * 0.5);
  while ((bi + 1) * (bi + 2) / 2 <= t) ++bi;
  while (bi * (bi + 1) / 2 > t) --bi;
  const int64_t bj = t - bi * (bi + 1) / 2;
  const int64_t i = bi * 16 + threadIdx.x / 16;
  const int64_t j = bj * 16 + threadIdx.x % 16;
  // gradient parts: lengthscales (gl), output scale (go), noise (gn); kept
  // apart so every register index is a compile-time constant
  double gl[BO_MAX_D];
#pragma unroll
  for (int e = 0; e < BO_MAX_D; ++e) gl[e] = 0.0;
  double go = 0.0, gn = 0.0;
  if (i < n && j < n && j <= i) {
    const double* ils = g.ils + k * d;
    const double s = g.os[k];
    const double a = alpha64[(int64_t)k * nf + i] * alpha64[(int64_t)k * nf + j] -
                     A[((int64_t)k * nf + i) * nf + j];
    const double wgt = (i == j) ? 0.5 : 1.0;     // 1/2 x (2 off the diagonal)
    double r2 = 0.0;
#pragma unroll
    for (int e = 0; e < BO_MAX_D; ++e) {
      if (e < d) {
        const double u = (static_cast<double>(X[i * d + e]) - static_cast<double>(X[j * d + e])) * ils[e];
        gl[e] = u * u;
        r2 += gl[e];
      }
    }
    const double r = sqrt(r2);
    const double c5 = 2.23606797749978969641;
    const double ex = exp(-c5 * r);
    const double common = wgt * a * (5.0 / 3.0) * s * (1.0 + c5 * r) * ex;
#pragma unroll
    for (int e = 0; e < BO_MAX_D; ++e) gl[e] *= common;   // 0 past d
    go = wgt * a * s * (1.0 + c5 * r + (5.0 / 3.0) * r2) * ex;
    gn = (i == j) ? 0.5 * a * g.noise[k] : 0.0;
  }
  // reduce the d + 2 sums over the workgroup
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int e = 0; e < BO_MAX_D + 2; ++e) {
    if (e < d || e >= BO_MAX_D) {
      double v = (e < BO_MAX_D) ? gl[e] : (e == BO_MAX_D ? go : gn);
      for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
      if (lane == 0) red[w][e < BO_MAX_D ? e : d + (e - BO_MAX_D)] = v;
    }
  }
  __syncthreads();
  if (threadIdx.x < d + 2) {
    const int e = threadIdx.x;
    partials[((int64_t)k * gridDim.x + t) * (d + 2) + e] =
        red[0][e] + red[1][e] + red[2][e] + red[3][e];
  }
}

// Sum of the per-tile gradient partials: one workgroup per (objective,
// gradient entry); each thread adds a strided subset of the tiles, then a
// fixed-shape tree over the workgroup (the order, so the result, does not
// depend on timing).
__global__ __launch_bounds__(256) void k_mll_reduce(const double* __restrict__ partials,
                                                    int64_t tiles, int d,
                                                    double* __restrict__ out) {
  __shared__ double red[256];
  const int k = blockIdx.x, e = blockIdx.y;
  double v = 0.0;
  for (int64_t t = threadIdx.x; t < tiles; t += 256)
    v += partials[((int64_t)k * tiles + t) * (d + 2) + e];
  red[threadIdx.x] = v;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[(int64_t)k * (d + 3) + 1 + e] = red[0];
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

// ---- noisy acquisition: in-sample posterior and its products --------------

// In-sample posterior covariance of the latent objective from K^{-1}:
// Sigma_XX = K_XX - K_XX K^{-1} K_XX = eta (I - eta K^{-1}) (K = K_XX + eta I,
// so K_XX = K - eta I). A holds K^{-1} in its lower 64-blocks on entry and
// Sigma_XX there on return, with an identity tail past n.
__global__ __launch_bounds__(256) void k_sigma_xx(double* __restrict__ A, int64_t n, int nf,
                                                  const double* __restrict__ noise) {
  const int k = blockIdx.y;
  const int t = blockIdx.x;
  int I = static_cast<int>((sqrt(8.0 * t + 1.0) - 1.0) * 0.5);
  while ((I + 1) * (I + 2) / 2 <= t) ++I;
  while (I * (I + 1) / 2 > t) --I;
  const int J = t - I * (I + 1) / 2;
  const double eta = noise[k];
  double* Ak = A + (int64_t)k * nf * nf;
  for (int e = threadIdx.x; e < B * B; e += 256) {
    const int64_t i = (int64_t)I * B + e / B, j = (int64_t)J * B + e % B;
    double* a = Ak + i * nf + j;
    if (i < n && j < n) *a = ((i == j) ? eta : 0.0) - eta * eta * *a;
    else *a = (i == j) ? 1.0 : 0.0;
  }
}

// Zk[k][i][s] = ZX[s][i][k] (fp64), zero for i >= n or s >= S.
__global__ __launch_bounds__(256) void k_gather_z(const float* __restrict__ ZX, int64_t n, int m,
                                                  int S, int nf, int Sp, double* __restrict__ Zk) {
  const int k = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)nf * Sp) return;
  const int64_t i = e / Sp;
  const int s = static_cast<int>(e % Sp);
  Zk[(int64_t)k * nf * Sp + e] =
      (i < n && s < S) ? static_cast<double>(ZX[((int64_t)s * n + i) * m + k]) : 0.0;
}

// C[k] = op(T[k]) Bm[k] for lower-triangular T [nf][nf] (only its lower
// 64-blocks are read; diagonal blocks hold zeros above the diagonal), op =
// identity or transpose; Bm, C [nf][ldb]. One 64x64 tile of C per workgroup,
// over the 64-blocks of T that the triangle leaves non-zero.
template <bool TRANS>
__global__ __launch_bounds__(256) void k_trmm(const double* __restrict__ T,
                                              const double* __restrict__ Bm,
                                              double* __restrict__ C, int nf, int ldb) {
  __shared__ double p[B][LDP];
  __shared__ double q[B][LDP];
  const int k = blockIdx.z, I = blockIdx.y, Jc = blockIdx.x;
  const int nbk = nf / B;
  const double* Tk = T + (int64_t)k * nf * nf;
  const double* Bk = Bm + (int64_t)k * nf * ldb;
  doublex4 acc[2][2] = {};
  const int k0 = TRANS ? I : 0, k1 = TRANS ? nbk : I + 1;
  for (int K = k0; K < k1; ++K) {
    __syncthreads();   // the previous step's tiles are no longer read
    double v0[16], v1[16];
    // P[i][t] = op(T)[I*B + i][K*B + t]; Q[c][t] = Bm[K*B + t][Jc*B + c]
    get_tile(v0, TRANS ? Tk + (int64_t)K * B * nf + I * B : Tk + (int64_t)I * B * nf + K * B, nf);
    get_tile(v1, Bk + (int64_t)K * B * ldb + Jc * B, ldb);
    put_tile<TRANS>(p, v0);
    put_tile<true>(q, v1);
    __syncthreads();
    gemm_nt_64(p, q, acc);
  }
  double* dst = C + (int64_t)k * nf * ldb + (int64_t)I * B * ldb + Jc * B;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 4; ++v) dst[(int64_t)tile_row(a, v) * ldb + tile_col(b)] = acc[a][b][v];
}

}  // namespace

hipError_t launch_gram(const float* X, int64_t n, int d, int m, int n_fit,
                       const GramParams& g, double* A, hipStream_t st,
                       unsigned long long* kdiag, int col0, int col1) {
  if (col1 < 0) col1 = n_fit;
  if (col0 % 16 != 0 || col1 % 16 != 0 || col0 < 0 || col1 > n_fit) return hipErrorInvalidValue;
  if (col1 <= col0) return hipSuccess;
  dim3 grid((col1 - col0) / 16, (n_fit + 15) / 16, m), block(16, 16);
  hipLaunchKernelGGL(k_gram, grid, block, 0, st, X, n, d, n_fit, g, A, kdiag, col0 / 16);
  return hipGetLastError();
}

hipError_t launch_weights(const float* X, int64_t n, int d, int m, int n_pad,
                          const GramParams& g, float* wts, hipStream_t st) {
  hipLaunchKernelGGL(k_weights, dim3((n_pad + 255) / 256, m), dim3(256), 0, st, X, n, d,
                     n_pad, g, wts);
  return hipGetLastError();
}

hipError_t launch_cholesky(double* A, double* W, int nf, int m, int* flag,
                           hipStream_t st, hipEvent_t before_update) {
  const int nbk = nf / B;
  hipLaunchKernelGGL(k_factor_first, dim3(m), dim3(kFactorThreads), 0, st, A, W, nf, flag);
  for (int kb = 0; kb < nbk; ++kb) {
    const int T = nbk - kb - 1;
    if (T + kb > 0)
      hipLaunchKernelGGL(k_panel, dim3(4 * (T + kb), m), dim3(256), 0, st, A, W, nf, kb);
    if (kb == 0 && before_update) {
      hipError_t e = hipStreamWaitEvent(st, before_update, 0);
      if (e != hipSuccess) return e;
    }
    if (T > 0)
      hipLaunchKernelGGL(k_update, dim3(T * (T + 1) / 2 + T * (kb + 1), m), dim3(kFactorThreads),
                         0, st, A, W, nf, kb, flag);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_alpha(const double* W, const float* Y, int64_t n, int m, int nf,
                        int n_pad, double* tmp, float* alpha, hipStream_t st,
                        double* alpha64) {
  hipLaunchKernelGGL(k_wy, dim3((nf + 3) / 4, m), dim3(256), 0, st, W, Y, n, m, nf, tmp);
  hipLaunchKernelGGL(k_wty, dim3((n_pad + 15) / 16, m), dim3(256), 0, st, W, tmp, n,
                     nf, n_pad, alpha, alpha64);
  return hipGetLastError();
}

int64_t mll_tiles(int nf) {
  const int64_t t = nf / 16;
  return t * (t + 1) / 2;
}

hipError_t launch_mll(const float* X, int64_t n, int d, int m, int nf, const GramParams& g,
                      double* A, const double* W, const double* tmp, const double* alpha64,
                      double* partials, double* out, hipStream_t st) {
  hipLaunchKernelGGL(k_logdet_quad, dim3(m), dim3(256), 0, st, A, tmp, n, nf, out, d);
  const int nbk = nf / B;
  hipLaunchKernelGGL(k_kinv, dim3(nbk * (nbk + 1) / 2, m), dim3(256), 0, st, A, W, nf);
  const int64_t tiles = mll_tiles(nf);
  hipLaunchKernelGGL(k_mll_grad, dim3(static_cast<unsigned>(tiles), m), dim3(256), 0, st, X, n,
                     d, nf, g, A, alpha64, partials);
  hipLaunchKernelGGL(k_mll_reduce, dim3(m, d + 2), dim3(256), 0, st, partials, tiles, d, out);
  return hipGetLastError();
}

hipError_t launch_scale_x(const float* X, int64_t n, int d, int m, int nb, int dx, int dr,
                          int dr4, const double* ils, float* invls, const double* pref_d,
                          float* pref, float* Xd, double* ils64, float* Xs, hipStream_t st) {
  const int n_pad = nb * kBlk;
  const unsigned gx2 = static_cast<unsigned>(((int64_t)n_pad * dx + 255) / 256);
  hipLaunchKernelGGL(k_scale_x, dim3(gx2, m), dim3(256), 0, st, X, n, d, dx, dr, dr4, n_pad,
                     ils, invls, pref_d, pref, d - dr, Xd, ils64, Xs);
  return hipGetLastError();
}

hipError_t launch_pack_x(const float* Xs, int64_t n, int m, int nb, int dx, int dr4,
                         float* ctr, uint16_t* xf, float* x2, hipStream_t st) {
  if (dx > 64 || n < 1) return hipErrorInvalidValue;
  const int n_pad = nb * kBlk;
  hipLaunchKernelGGL(k_center_x, dim3(dx, m), dim3(256), 0, st, Xs, n, n_pad, dx, ctr);
  const int64_t th = (int64_t)nb * dist_frags(dx) * 64;
  hipLaunchKernelGGL(k_pack_x, dim3(static_cast<unsigned>((th + 255) / 256), m), dim3(256), 0, st,
                     Xs, n, n_pad, nb, dx, ctr, reinterpret_cast<_Float16*>(xf));
  hipLaunchKernelGGL(k_norm_x, dim3(static_cast<unsigned>((n_pad + 255) / 256), m), dim3(256), 0,
                     st, Xs, n, n_pad, dx, dr4, ctr, x2);
  return hipGetLastError();
}

hipError_t launch_kinv(double* A, const double* W, int nf, int m, hipStream_t st) {
  const int nbk = nf / B;
  hipLaunchKernelGGL(k_kinv, dim3(nbk * (nbk + 1) / 2, m), dim3(256), 0, st, A, W, nf);
  return hipGetLastError();
}

hipError_t launch_sigma_xx(double* A, int64_t n, int nf, int m, const double* noise,
                           hipStream_t st) {
  const int nbk = nf / B;
  hipLaunchKernelGGL(k_sigma_xx, dim3(nbk * (nbk + 1) / 2, m), dim3(256), 0, st, A, n, nf, noise);
  return hipGetLastError();
}

hipError_t launch_gather_z(const float* ZX, int64_t n, int m, int S, int nf, int Sp,
                           double* Zk, hipStream_t st) {
  const unsigned g = static_cast<unsigned>(((int64_t)nf * Sp + 255) / 256);
  hipLaunchKernelGGL(k_gather_z, dim3(g, m), dim3(256), 0, st, ZX, n, m, S, nf, Sp, Zk);
  return hipGetLastError();
}

hipError_t launch_trmm(bool trans, const double* T, const double* Bm, double* C, int nf,
                       int ldb, int m, hipStream_t st) {
  if (nf % B != 0 || ldb % B != 0) return hipErrorInvalidValue;
  const dim3 grid(ldb / B, nf / B, m);
  if (trans) hipLaunchKernelGGL(k_trmm<true>, grid, dim3(256), 0, st, T, Bm, C, nf, ldb);
  else hipLaunchKernelGGL(k_trmm<false>, grid, dim3(256), 0, st, T, Bm, C, nf, ldb);
  return hipGetLastError();
}

hipError_t launch_pack_factor(const double* W, int64_t n, int m, int nf, int nb, float* Lp,
                              unsigned long long* wmax, int* flag, hipStream_t st,
                              unsigned long long* bmax) {
  const int64_t nblk = posterior_frag_blocks(nb);   // with the zero block
  const int64_t stride = static_cast<int64_t>(packed_factor_floats(nb));
  float* rsc = Lp + nblk * 512;                     // objective k's scales at rsc + k * stride
  if (bmax) {
    const unsigned nch = static_cast<unsigned>((n + 255) / 256);
    hipLaunchKernelGGL(k_rowblock_max, dim3(nb, nch, m), dim3(256), 0, st, W, n, nf, nb, bmax,
                       flag);
  } else {
    hipLaunchKernelGGL(k_rowblock_scale, dim3(nb, m), dim3(256), 0, st, W, n, nf, rsc, stride,
                       wmax, flag);
  }
  const unsigned gx = static_cast<unsigned>((nblk * 64 + 255) / 256);
  hipLaunchKernelGGL(k_pack, dim3(gx, m), dim3(256), 0, st, W, n, nf, nblk, nb, rsc, stride,
                     reinterpret_cast<_Float16*>(Lp), static_cast<const unsigned long long*>(bmax),
                     wmax);
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
