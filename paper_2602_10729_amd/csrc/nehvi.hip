// Noisy expected hypervolume improvement (qNEHVI; q-batches, two or three objectives).
//
// Paper: "Overall MOBO workflow" step (ii) and the constrained qNEHVI
// paragraph: the acquisition averages, over Monte-Carlo samples of the joint
// posterior, the hypervolume improvement of the candidate; the noisy form
// (after Daulton et al. 2021) samples the latent objectives at the observed
// points too and measures each sample's improvement against the Pareto front
// of that sample's in-sample values.
//
// Given the in-sample draw f_X^s, the candidate's latent value is Gaussian
// with mean k*^T K_XX^{-1} f_X^s and variance tau^2 = s - k*^T K_XX^{-1} k*
// (once f_X is known the noisy y adds nothing, so this is the noise-free GP).
// With f_X^s = mu_X + L_XX z_X^s (L_XX the factor of the in-sample posterior
// covariance) and K_XX^{-1} mu_X = K^{-1} y:
//   y_s = mu* + (K* G)[s] + tau z*_s,   G = K_XX^{-1} L_XX Z_X  [n][S],
// mu* the ordinary posterior mean.
//
// bo_nehvi_prepare (fp64, once per set of in-sample base samples) builds
// f_X^s, every sample's front and staircase boxes (k_sample_front for two
// objectives; k_insample_values and k_sample_front3 for three), G and its
// fp16 hi/lo fragments (k_pack_g), and the packed inverse factor of K_XX.
// Scoring runs per chunk of candidates: the posterior kernel on the
// noise-free factor (mu*, tau), k_nehvi_means (K* G on the matrix cores, K*
// evaluated on the fly), then k_nehvi_ehvi (per-sample HVI against that
// sample's boxes).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "bo_internal.h"
#include "kv_scale.h"

namespace bo {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef _Float16 halfx4 __attribute__((ext_vector_type(4)));

// ---- per-sample fronts --------------------------------------------------------

// One workgroup per sample s. In-sample values
//   f_ik = y_ik - eta_k alpha_k,i + (L_XX Z_X)[k][i][s]   (mu_X = y - eta alpha),
// points strictly above ref (and meeting the feasibility thresholds) take
// part; the front is the non-dominated set (maximise; exact duplicates keep
// the lowest index), sorted by objective 0 ascending. Box r (r < P) spans
// objective 0 from the previous front value (ref for r = 0) to f_r,0 and
// objective 1 from f_r,1 up; box P spans objective 0 from the last front
// value up and objective 1 from ref up. Boxes are (lo0, lo1, width0, width1),
// widths in fp32 (inf for unbounded sides).
__global__ __launch_bounds__(256) void k_sample_front(NehviFrontArgs a) {
  extern __shared__ double fsh[];
  __shared__ int tsum[256];
  __shared__ int np;
  const int n = static_cast<int>(a.n);
  double* f0 = fsh;
  double* f1 = fsh + n;
  int* flag = reinterpret_cast<int*>(fsh + 2 * n);
  int* pidx = flag + n;
  int* sorted = pidx + n;
  const int s = blockIdx.x, tid = threadIdx.x;
  const double e0 = a.noise[0], e1 = a.noise[1];
  for (int i = tid; i < n; i += 256) {
    const double v0 = static_cast<double>(a.Y[2 * i]) - e0 * a.alpha64[i] +
                      a.T1[(int64_t)i * a.Sp + s];
    const double v1 = static_cast<double>(a.Y[2 * i + 1]) - e1 * a.alpha64[a.nf + i] +
                      a.T1[((int64_t)a.nf + i) * a.Sp + s];
    bool ok = v0 > static_cast<double>(a.ref0) && v1 > static_cast<double>(a.ref1);
    if (a.cons) ok = ok && v0 >= static_cast<double>(a.low0) && v1 >= static_cast<double>(a.low1);
    // points that take no part can dominate nothing
    f0[i] = ok ? v0 : -__builtin_inf();
    f1[i] = ok ? v1 : -__builtin_inf();
    flag[i] = ok ? 1 : 0;
  }
  __syncthreads();
  for (int i = tid; i < n; i += 256) {
    if (!flag[i]) continue;
    const double a0 = f0[i], a1 = f1[i];
    bool dom = false;
    for (int j = 0; j < n; ++j) {
      const double b0 = f0[j], b1 = f1[j];
      const bool ge = b0 >= a0 && b1 >= a1;
      dom = dom || (ge && (b0 > a0 || b1 > a1)) || (ge && b0 == a0 && b1 == a1 && j < i);
    }
    pidx[i] = dom ? 0 : 1;          // front flags (flag[] is still read by others)
  }
  __syncthreads();
  for (int i = tid; i < n; i += 256) flag[i] = flag[i] ? pidx[i] : 0;
  __syncthreads();
  // compaction in index order: thread t owns a contiguous chunk
  const int per = (n + 255) / 256;
  const int i0 = min(n, tid * per), i1 = min(n, i0 + per);
  int cnt = 0;
  for (int i = i0; i < i1; ++i) cnt += flag[i];
  tsum[tid] = cnt;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int t = 0; t < 256; ++t) {
      const int c = tsum[t];
      tsum[t] = run;
      run += c;
    }
    np = run;
  }
  __syncthreads();
  {
    int p = tsum[tid];
    for (int i = i0; i < i1; ++i)
      if (flag[i]) pidx[p++] = i;
  }
  __syncthreads();
  const int P = np;
  // rank by objective 0 (ties by position, i.e. by index)
  for (int q = tid; q < P; q += 256) {
    const double v = f0[pidx[q]];
    int rank = 0;
    for (int r = 0; r < P; ++r) {
      const double w = f0[pidx[r]];
      rank += (w < v || (w == v && r < q)) ? 1 : 0;
    }
    sorted[rank] = pidx[q];
  }
  __syncthreads();
  float* bx = a.boxes + (int64_t)s * (n + 1) * 4;
  for (int r = tid; r <= P; r += 256) {
    float lo0, lo1, w0, w1 = __builtin_inff();
    lo0 = (r == 0) ? a.ref0 : static_cast<float>(f0[sorted[r - 1]]);
    if (r < P) {
      const int i = sorted[r];
      w0 = static_cast<float>(f0[i]) - lo0;
      lo1 = static_cast<float>(f1[i]);
      a.front[(int64_t)s * n + r] = i;
    } else {
      w0 = __builtin_inff();
      lo1 = a.ref1;
    }
    *reinterpret_cast<float4*>(bx + 4 * r) = float4{lo0, lo1, w0, w1};
  }
  if (tid == 0) a.counts[s] = P + 1;
}

// Three objectives, one workgroup per sample s, from the in-sample values
// F[s][i][k] (fp64). The front is selected by the rule above (points
// strictly above ref and meeting the thresholds; non-dominated, exact
// duplicates keep the lowest index) and listed by objective 0 ascending
// (ties by index). Its boxes come from a sweep over the front points by
// objective 2 descending (ties in list order) that keeps the staircase of
// the points swept so far in the (objective 0, objective 1) plane, sorted by
// objective 0: step t covers objective 0 from the previous step's value (ref
// for the first) to its own and objective 1 from its own value up, and
// carries the objective-2 value where its current box began (its top). A
// new point that lies under a step in both coordinates adds nothing; else it
// removes the steps it covers (objective 0 and 1 both at most its own), each
// removed step and the step to its right (or the tail box past the last
// step) close a box from the new point's objective 2 up to their tops, and it
// enters the staircase with its own value as top; the step to its right
// restarts there too. After the sweep every step, and the tail box above
// ref_1, closes down to ref_2. Boxes are (lo0, lo1, lo2, w0, w1, w2) with
// widths in fp32 (inf for unbounded sides), at most 3P + 1 per sample:
// boxes[s][3n + 1][6], counts[s] = their number, counts[S + s] = P; a
// non-finite value sets *bad.
__global__ __launch_bounds__(256) void k_sample_front3(NehviFront3Args a) {
  extern __shared__ double fsh[];
  __shared__ int tsum[256];
  __shared__ int np;
  const int n = static_cast<int>(a.n);
  double* f0 = fsh;
  double* f1 = f0 + n;
  double* f2 = f1 + n;
  double* sx = f2 + n;          // staircase: objective 0, 1, top
  double* sy = sx + n;
  double* sz = sy + n;
  int* flag = reinterpret_cast<int*>(sz + n);
  int* pidx = flag + n;
  int* sorted = pidx + n;
  const int s = blockIdx.x, tid = threadIdx.x;
  const double r0 = a.ref[0], r1 = a.ref[1], r2 = a.ref[2];
  bool bad = false;
  for (int i = tid; i < n; i += 256) {
    const double* v = a.F + ((int64_t)s * n + i) * 3;
    const double v0 = v[0], v1 = v[1], v2 = v[2];
    bad = bad || !(fabs(v0) < __builtin_inf() && fabs(v1) < __builtin_inf() &&
                   fabs(v2) < __builtin_inf());
    bool ok = v0 > r0 && v1 > r1 && v2 > r2;
    if (a.cons)
      ok = ok && v0 >= static_cast<double>(a.low[0]) && v1 >= static_cast<double>(a.low[1]) &&
           v2 >= static_cast<double>(a.low[2]);
    f0[i] = ok ? v0 : -__builtin_inf();
    f1[i] = ok ? v1 : -__builtin_inf();
    f2[i] = ok ? v2 : -__builtin_inf();
    flag[i] = ok ? 1 : 0;
  }
  if (bad) atomicOr(a.bad, 1);
  // j beats i: at least as large in every objective and larger in one, or an
  // exact duplicate with a lower index (a strict order: the front is the set
  // of points nothing beats)
  auto beats = [&](int j, int i) {
    const double a0 = f0[i], a1 = f1[i], a2 = f2[i], b0 = f0[j], b1 = f1[j], b2 = f2[j];
    return b0 >= a0 && b1 >= a1 && b2 >= a2 && (b0 > a0 || b1 > a1 || b2 > a2 || j < i);
  };
  // compaction of the flagged points in index order into pidx (thread t owns
  // a contiguous chunk); returns their number
  const int per = (n + 255) / 256;
  const int i0 = min(n, tid * per), i1 = min(n, i0 + per);
  auto compact = [&]() {
    __syncthreads();
    int cnt = 0;
    for (int i = i0; i < i1; ++i) cnt += flag[i];
    tsum[tid] = cnt;
    __syncthreads();
    if (tid == 0) {
      int run = 0;
      for (int t = 0; t < 256; ++t) {
        const int c = tsum[t];
        tsum[t] = run;
        run += c;
      }
      np = run;
    }
    __syncthreads();
    int p = tsum[tid];
    for (int i = i0; i < i1; ++i)
      if (flag[i]) pidx[p++] = i;
    __syncthreads();
    return np;
  };
  // Screen: the largest-sum point of each thread's chunk forms a strong set;
  // a point some member beats is not on the front. Then the survivors are
  // checked against each other: a point off the front is beaten by a front
  // point (the order is transitive), and front points survive the screen.
  {
    int best = -1;
    double bs = -__builtin_inf();
    for (int i = i0; i < i1; ++i) {
      const double sm = f0[i] + f1[i] + f2[i];
      if (flag[i] && sm > bs) {
        bs = sm;
        best = i;
      }
    }
    __syncthreads();
    tsum[tid] = best;
    __syncthreads();
    for (int i = tid; i < n; i += 256) {
      if (!flag[i]) continue;
      bool dom = false;
      for (int t = 0; t < 256 && !dom; ++t) {
        const int j = tsum[t];
        dom = j >= 0 && beats(j, i);
      }
      pidx[i] = dom ? 0 : 1;
    }
    __syncthreads();
    for (int i = tid; i < n; i += 256) flag[i] = flag[i] ? pidx[i] : 0;
  }
  const int V = compact();                     // survivors in pidx[0, V)
  for (int q = tid; q < V; q += 256) sorted[q] = pidx[q];
  __syncthreads();
  for (int q = tid; q < V; q += 256) {
    const int i = sorted[q];
    bool dom = false;
    for (int r = 0; r < V && !dom; ++r) dom = beats(sorted[r], i);
    flag[i] = dom ? 0 : 1;
  }
  const int P = compact();
  // list order: objective 0 ascending, ties by index
  for (int q = tid; q < P; q += 256) {
    const double v = f0[pidx[q]];
    int rank = 0;
    for (int r = 0; r < P; ++r) {
      const double w = f0[pidx[r]];
      rank += (w < v || (w == v && r < q)) ? 1 : 0;
    }
    sorted[rank] = pidx[q];
    a.front[(int64_t)s * n + rank] = pidx[q];
  }
  __syncthreads();
  // sweep order: objective 2 descending, ties in list order (flag[] reused)
  for (int q = tid; q < P; q += 256) {
    const double v = f2[sorted[q]];
    int rank = 0;
    for (int r = 0; r < P; ++r) {
      const double w = f2[sorted[r]];
      rank += (w > v || (w == v && r < q)) ? 1 : 0;
    }
    flag[rank] = sorted[q];
  }
  __syncthreads();
  if (tid != 0) return;
  float* bx = a.boxes + (int64_t)s * (3 * n + 1) * 6;
  int nb = 0;
  auto close = [&](double xl, double xh, double yl, double zl, double zt) {
    if (zt > zl) {
      const float l0 = static_cast<float>(xl), l1 = static_cast<float>(yl),
                  l2 = static_cast<float>(zl);
      float* o = bx + 6 * nb;
      o[0] = l0;
      o[1] = l1;
      o[2] = l2;
      o[3] = static_cast<float>(xh) - l0;
      o[4] = __builtin_inff();
      o[5] = static_cast<float>(zt) - l2;
      ++nb;
    }
  };
  int cntst = 0;
  double tail = __builtin_inf();
  for (int t = 0; t < P; ++t) {
    const int idx = flag[t];
    const double px = f0[idx], py = f1[idx], zb = f2[idx];
    int p = 0, hi = cntst;                       // first step with x >= px
    while (p < hi) {
      const int mid = (p + hi) >> 1;
      if (sx[mid] < px) p = mid + 1;
      else hi = mid;
    }
    if (p < cntst && sy[p] >= py) continue;      // under a step in both coordinates
    const int first_rm = (p < cntst && sx[p] == px) ? p + 1 : p;
    int left = p;
    while (left > 0 && sy[left - 1] <= py) --left;
    double xl = (left == 0) ? r0 : sx[left - 1];
    for (int r = left; r < first_rm; ++r) {
      close(xl, sx[r], sy[r], zb, sz[r]);
      xl = sx[r];
    }
    if (first_rm < cntst) {
      close(xl, sx[first_rm], sy[first_rm], zb, sz[first_rm]);
      sz[first_rm] = zb;
    } else {
      close(xl, __builtin_inf(), r1, zb, tail);
      tail = zb;
    }
    // steps [left, first_rm) give way to the new one at left
    const int removed = first_rm - left;
    if (removed == 0) {
      for (int r = cntst; r > left; --r) {
        sx[r] = sx[r - 1];
        sy[r] = sy[r - 1];
        sz[r] = sz[r - 1];
      }
    } else {
      for (int r = first_rm; r < cntst; ++r) {
        sx[r - removed + 1] = sx[r];
        sy[r - removed + 1] = sy[r];
        sz[r - removed + 1] = sz[r];
      }
    }
    cntst += 1 - removed;
    sx[left] = px;
    sy[left] = py;
    sz[left] = zb;
  }
  double xl = r0;
  for (int r = 0; r < cntst; ++r) {
    close(xl, sx[r], sy[r], r2, sz[r]);
    xl = sx[r];
  }
  close(xl, __builtin_inf(), r1, r2, tail);
  a.counts[s] = nb;
  a.counts[a.S + s] = P;
}

// Boxes of three objectives from [S][stride] to the compact layout at off[s].
__global__ __launch_bounds__(64) void k_compact_boxes3(const float* __restrict__ tmp,
                                                       int64_t stride, const int* __restrict__ off,
                                                       float* __restrict__ out) {
  const int s = blockIdx.x;
  const int b0 = off[s], nb = off[s + 1] - b0;
  for (int e = threadIdx.x; e < 6 * nb; e += 64) out[6 * (int64_t)b0 + e] = tmp[(int64_t)s * stride + e];
}

// part[k][b] = max |G[k][e]| over the entries e = b*256 + t (mod 256 x
// gridDim.x) of workgroup b; the host takes the maximum of the parts.
__global__ __launch_bounds__(256) void k_absmax(const double* __restrict__ G, int64_t count,
                                                double* __restrict__ part) {
  __shared__ double red[256];
  const int k = blockIdx.y;
  const double* g = G + (int64_t)k * count;
  double v = 0.0;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < count; e += (int64_t)gridDim.x * 256)
    v = fmax(v, fabs(g[e]));
  red[threadIdx.x] = v;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (threadIdx.x < h) red[threadIdx.x] = fmax(red[threadIdx.x], red[threadIdx.x + h]);
    __syncthreads();
  }
  if (threadIdx.x == 0) part[(int64_t)k * gridDim.x + blockIdx.x] = red[0];
}

// The in-sample draws f_ik = y_ik - eta_k alpha_k,i + T1[k][i][s] (mu_X =
// y - eta alpha) as F [S][n][m], fp64, for the host's per-draw fronts.
__global__ __launch_bounds__(256) void k_insample_values(const float* __restrict__ Y,
                                                         const double* __restrict__ alpha64,
                                                         const double* __restrict__ noise,
                                                         const double* __restrict__ T1,
                                                         int64_t n, int m, int nf, int Sp, int S,
                                                         double* __restrict__ F) {
  const int k = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;   // s * n + i
  if (e >= (int64_t)S * n) return;
  const int64_t i = e % n;
  const int s = static_cast<int>(e / n);
  F[e * m + k] = static_cast<double>(Y[i * m + k]) - noise[k] * alpha64[(int64_t)k * nf + i] +
                 T1[((int64_t)k * nf + i) * Sp + s];
}

// A fragments of G^T (scaled by sc[k]) for v_mfma_f32_16x16x32_f16: block
// (J, rb) covers training rows 32J .. 32J+31 and samples 16rb .. 16rb+15;
// lane l element e holds G[32J + 8(l/16) + e][16rb + l%16], split as
// hi = fp16(g), lo = fp16(g - hi). Layout [k][J][rb][plane][64][8].
__global__ __launch_bounds__(256) void k_pack_g(const double* __restrict__ G, int nf, int Sp,
                                                int n32, int nrb, float sc0, float sc1,
                                                float sc2, _Float16* __restrict__ Gp) {
  const int k = blockIdx.y;
  const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (g >= (int64_t)n32 * nrb * 64) return;
  const int lane = static_cast<int>(g % 64);
  const int64_t blk = g / 64;
  const int J = static_cast<int>(blk / nrb), rb = static_cast<int>(blk % nrb);
  const double sc = (k == 0) ? sc0 : (k == 1) ? sc1 : sc2;
  const int col = 16 * rb + lane % 16;
  _Float16* dst = Gp + ((int64_t)k * n32 * nrb + blk) * 1024 + lane * 8;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int row = 32 * J + 8 * (lane / 16) + e;
    const double w = sc * G[((int64_t)k * nf + row) * Sp + col];
    const _Float16 h = static_cast<_Float16>(static_cast<float>(w));
    dst[e] = h;
    dst[512 + e] = static_cast<_Float16>(static_cast<float>(w - static_cast<double>(h)));
  }
}

// Boxes of sample s from the per-sample layout [S][stride] to the compact
// one at off[s].
__global__ __launch_bounds__(64) void k_compact_boxes(const float* __restrict__ tmp,
                                                      int64_t stride, const int* __restrict__ off,
                                                      float* __restrict__ out) {
  const int s = blockIdx.x;
  const int b0 = off[s], nb = off[s + 1] - b0;
  for (int b = threadIdx.x; b < nb; b += 64)
    *reinterpret_cast<float4*>(out + 4 * (int64_t)(b0 + b)) =
        *reinterpret_cast<const float4*>(tmp + (int64_t)s * stride + 4 * b);
}

// ---- conditional means K* G on the matrix cores -------------------------------

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}

__device__ __forceinline__ float4 ld4(__amdgpu_buffer_rsrc_t rs, int voff, int soff) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, soff, 0));
}

// LDS-only barrier: waits for this wave's LDS traffic, not for its global
// loads in flight (the next step's fragments), then joins the workgroup.
__device__ __forceinline__ void lds_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ float m32(float r2) {
  const float r = __builtin_amdgcn_sqrtf(r2);
  constexpr float kNegSqrt3Log2e = static_cast<float>(-1.73205080756887729353 * 1.44269504088896340736);
  return fmaf(r, 1.73205081f, 1.0f) * __builtin_amdgcn_exp2f(kNegSqrt3Log2e * r);
}

__device__ __forceinline__ float m52(float r2, float s) {
  const float r = __builtin_amdgcn_sqrtf(r2);
  constexpr float kNegSqrt5Log2e = static_cast<float>(-2.23606797749978969641 * 1.44269504088896340736);
  const float e = __builtin_amdgcn_exp2f(kNegSqrt5Log2e * r);
  return s * fmaf(r, 2.23606798f, fmaf(r2, 1.66666667f, 1.0f)) * e;
}

constexpr int kMW = 8;                 // waves per workgroup
constexpr int kMT = 64;                // candidates per tile
constexpr int kKS = 40;                // ring: halves per candidate row (32 + 8 pad)
constexpr int kPlane = kMT * kKS;      // halves per fp16 plane
constexpr int kRingSlot = 2 * kPlane;  // hi + lo planes of one 32-row block

// D[k][s][c] = sum_i G[k][i][s] K*_k(c, i) for the candidates of one tile and
// every sample: blockIdx.x = tile of 64 candidates, blockIdx.y = objective.
// Each 32-row block J of K*^T (training rows x candidates) is evaluated two
// steps ahead into a three-slot LDS ring as fp16 hi/lo planes, while the
// matrix cores add G^T[slots of this wave][J] K*^T[J] into accumulators that
// stay in registers for the whole tile: wave w owns the sample blocks w + 8r
// (r < CB), all four candidate blocks. Three products per pair (hi hi, hi lo,
// lo hi), fp32 accumulate. Training rows past the matrix read as zero; their
// G rows are zero, so they add nothing.
// The kernel values are made as the posterior kernel makes them: wave w
// forms the squared distances of rows 16(w/4) .. +15 and candidates
// 16(w%4) .. +15 of a block with a few more MFMAs (|c|^2 + |x|^2 - 2 c.x over
// centred coordinates, from the training rows' distance fragments the fit
// stores and the candidates' made here), and recomputes a pair from exact
// differences of the scaled coordinates where the expansion could cancel
// (approximate r^2 below 1 + (|c|^2 + |x|^2)/256). COMP: the composite kernel
//   s_route M52(r_route) + s_dep w(c) w(x) M32(r_dep) + s_int M52 M32,
// one expansion per coordinate group (routing slots first).
template <int DX4, int CB, bool COMP>
__global__ __launch_bounds__(kMW * 64) void k_nehvi_means(NehviMeansArgs a) {
  constexpr int RS = 4 * DX4;
  constexpr int NS = COMP ? 2 : 1;
  constexpr int F0 = dist_frags0(RS), NF = dist_frags(RS);
  static_assert(F0 == 1 && NF <= 3, "at most 32 coordinate slots");
  static_assert(2 * kMT * 96 <= 3 * kRingSlot, "candidate fragments fit the ring");
  __shared__ __align__(16) _Float16 ring[3 * kRingSlot];
  __shared__ __align__(16) float ctile[kMT * RS];   // exact scaled candidates
  __shared__ float kish[kMT];              // 2^(E-14): undoes a candidate's split scale
  const int k = blockIdx.y;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t c0 = (int64_t)blockIdx.x * kMT;
  const int nrb = 8 * CB;
  const float* il = a.invls + k * a.dx;
  const float* ctr = a.ctr + k * a.dx;
  const float sk = a.s[k];
  const float sint = COMP ? a.s_int[k] : 0.f;
  const __amdgpu_buffer_rsrc_t xs_rs = rsrc(a.Xs + (int64_t)k * a.n_pad * a.dx,
                                            a.n_pad * a.dx * 4);
  const __amdgpu_buffer_rsrc_t xf_rs = rsrc(a.xf + (int64_t)k * a.xf_stride,
                                            (a.n_pad / 16) * NF * 1024);
  const __amdgpu_buffer_rsrc_t x2_rs = rsrc(a.x2 + (int64_t)k * 2 * a.n_pad, 2 * a.n_pad * 4);
  const __amdgpu_buffer_rsrc_t w_rs = rsrc(COMP ? a.wts + (int64_t)k * a.n_pad : a.Xs,
                                           COMP ? a.n_pad * 4 : 0);
  const __amdgpu_buffer_rsrc_t g_rs = rsrc(a.Gp + (int64_t)k * a.n32 * nrb * 1024,
                                           a.n32 * nrb * 2048);
  // this lane's place in a produced block: column (candidate) col, rows
  // rq .. rq+3 (the MFMA result layout of its wave's 16x16 distance tile)
  const int half = wave >> 2;
  const int col = 16 * (wave & 3) + (lane & 15);
  const int rq = 16 * half + 4 * (lane >> 4);
  // the column's candidate, scaled, in the slot layout (zero past npts and in
  // padding slots); COMP: s_dep times its preference weight
  float cc[RS];
  float wsd = 0.f, wstar = 0.f;
  {
    const int64_t c = c0 + col;
    const bool ok = c < a.npts;
#pragma unroll
    for (int t = 0; t < RS; ++t) {
      const int cd = slot_dim(t, a.d, a.dr, a.dr4);
      cc[t] = (ok && cd >= 0) ? a.cand[c * a.d + cd] * il[t] : 0.f;
    }
    if constexpr (COMP) {
      if (ok) {
        const float* pr = a.pref + (int64_t)k * (a.d - a.dr);
        float e = 0.f;
        for (int t = a.dr; t < a.d; ++t) e = fmaf(pr[t - a.dr], a.cand[c * a.d + t], e);
        wstar = expf(e);
        wsd = a.s_dep[k] * wstar;
      }
    }
  }
  // power of two for this column's kernel values before their split (the
  // composite covariance is bounded by sqrt(prior(candidate) * kbound)); the
  // values are made scaled, the scale rides in the output scales
  const KvScale ks = kv_split_scale(
      COMP ? __builtin_amdgcn_sqrtf(fmaf(wsd, wstar, sk + sint) * a.kbound[k]) : sk);
  const float sks = sk * ks.ksc, sints = sint * ks.ksc;
  wsd *= ks.ksc;
  // centred coordinates: squared norms per group, and the B fragments of the
  // distance MFMAs, staged in the (not yet used) ring as 96 halves per group
  // and column: [0, 32) stream 0 (hi, zero past RS), [32, 96) stream 1 (hi at
  // p < RS, 2^11-scaled lo at RS <= p < 2RS, zero beyond)
  float c2[NS];
  halfx8 cb[NS][NF];
  {
    float ct[RS];
#pragma unroll
    for (int t = 0; t < RS; ++t) ct[t] = cc[t] - ctr[t];
#pragma unroll
    for (int g = 0; g < NS; ++g) {
      float n2 = 0.f;
#pragma unroll
      for (int t = 0; t < RS; ++t) {
        const bool in = !COMP || ((t < 4 * a.dr4) == (g == 0));
        if (in) n2 = fmaf(ct[t], ct[t], n2);
      }
      c2[g] = n2;
    }
    if (half == 0 && (lane >> 4) == 0) {
#pragma unroll
      for (int g = 0; g < NS; ++g) {
        _Float16* h = ring + (g * kMT + col) * 96;
        halfx8 v[12];
#pragma unroll
        for (int i = 0; i < 12; ++i) v[i] = halfx8{};
#pragma unroll
        for (int t = 0; t < RS; ++t) {
          const bool in = !COMP || ((t < 4 * a.dr4) == (g == 0));
          const _Float16 hi = static_cast<_Float16>(in ? ct[t] : 0.f);
          const _Float16 lo = static_cast<_Float16>(
              in ? (ct[t] - static_cast<float>(static_cast<_Float16>(ct[t]))) * kDistLoScale : 0.f);
          v[t / 8][t % 8] = hi;
          v[(32 + t) / 8][(32 + t) % 8] = hi;
          v[(32 + RS + t) / 8][(32 + RS + t) % 8] = lo;
        }
#pragma unroll
        for (int i = 0; i < 12; ++i) *reinterpret_cast<halfx8*>(h + 8 * i) = v[i];
      }
#pragma unroll
      for (int t4 = 0; t4 < DX4; ++t4)
        *reinterpret_cast<float4*>(ctile + col * RS + 4 * t4) =
            float4{cc[4 * t4], cc[4 * t4 + 1], cc[4 * t4 + 2], cc[4 * t4 + 3]};
      kish[col] = ks.kinv;
    }
    __syncthreads();
#pragma unroll
    for (int g = 0; g < NS; ++g)
#pragma unroll
      for (int f = 0; f < NF; ++f)
        cb[g][f] = *reinterpret_cast<const halfx8*>(ring + (g * kMT + col) * 96 + 32 * f +
                                                    8 * (lane >> 4));
    __syncthreads();   // the ring is written from here on
  }

  // operands of the block made next, loaded a step ahead
  halfx8 xa[NF];
  floatx4 x2v[NS], wtv;
  auto prod_load = [&](int jb) {
    const int vo = (2 * jb + half) * (NF * 1024) + lane * 16;
#pragma unroll
    for (int f = 0; f < NF; ++f) xa[f] = __builtin_bit_cast(halfx8, ld4(xf_rs, vo + f * 1024, 0));
    const int row = jb * 32 + rq;
#pragma unroll
    for (int g = 0; g < NS; ++g)
      x2v[g] = __builtin_bit_cast(floatx4, ld4(x2_rs, ((COMP ? g : 1) * a.n_pad + row) * 4, 0));
    if constexpr (COMP) wtv = __builtin_bit_cast(floatx4, ld4(w_rs, row * 4, 0));
  };
  auto produce = [&](int jb) {
    floatx4 d0[NS], d1[NS];
#pragma unroll
    for (int g = 0; g < NS; ++g) {
      d0[g] = floatx4{0.f, 0.f, 0.f, 0.f};
      d1[g] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int f = 0; f < F0; ++f)
        d0[g] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[f], cb[g][f], d0[g], 0, 0, 0);
#pragma unroll
      for (int f = F0; f < NF; ++f)
        d1[g] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[f], cb[g][f], d1[g], 0, 0, 0);
    }
    float r2[NS][4];
    bool ex[4];
    bool any = false;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float rt = 0.f, nt = 0.f;
#pragma unroll
      for (int g = 0; g < NS; ++g) {
        const float nrm = c2[g] + x2v[g][e];
        const float dot = fmaf(d1[g][e], 1.0f / kDistLoScale, d0[g][e]);
        r2[g][e] = fmaxf(fmaf(-2.0f, dot, nrm), 0.f);
        rt += r2[g][e];
        nt += nrm;
      }
      ex[e] = rt < fmaf(nt, 1.0f / 256.0f, 1.0f);
      any = any || ex[e];
    }
    if (__builtin_amdgcn_ballot_w64(any) != 0) {
      // exact differences for the pairs that need them (rows past n_pad read
      // zero coordinates); rare, kept off the common path
      asm volatile("" ::: "memory");
      const float* cx = ctile + col * RS;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = jb * 32 + rq + e;
        float s0 = 0.f, s1 = 0.f;   // routing / deployment (plain: s1 only)
#pragma unroll
        for (int t4 = 0; t4 < DX4; ++t4) {
          const float4 x = ld4(xs_rs, (row * a.dx + 4 * t4) * 4, 0);
          const float4 cv = *reinterpret_cast<const float4*>(cx + 4 * t4);
          const float e0 = cv.x - x.x, e1 = cv.y - x.y, e2 = cv.z - x.z, e3 = cv.w - x.w;
          float t = fmaf(e0, e0, 0.f);
          t = fmaf(e1, e1, t);
          t = fmaf(e2, e2, t);
          t = fmaf(e3, e3, t);
          if (COMP && t4 < a.dr4) s0 += t;
          else s1 += t;
        }
        if (ex[e]) {
          if constexpr (COMP) {
            r2[0][e] = s0;
            r2[1][e] = s1;
          } else {
            r2[0][e] = s1;
          }
        }
      }
    }
    halfx4 hi, lo;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float kv;
      if constexpr (COMP) {
        const float k5 = m52(r2[0][e], 1.0f);
        const float k3 = m32(r2[1][e]);
        kv = fmaf(wsd * wtv[e], k3, k5 * fmaf(sints, k3, sks));
      } else {
        kv = m52(r2[0][e], sks);
      }
      // one fp32 value for both halves (the compiler may otherwise fuse the
      // last product into the fp16 conversions and derive the high half twice)
      asm volatile("" : "+v"(kv));
      const _Float16 h = static_cast<_Float16>(kv);
      hi[e] = h;
      lo[e] = static_cast<_Float16>(kv - static_cast<float>(h));
    }
    _Float16* dst = ring + (jb % 3) * kRingSlot + col * kKS + rq;
    *reinterpret_cast<halfx4*>(dst) = hi;
    *reinterpret_cast<halfx4*>(dst + kPlane) = lo;
  };
  auto load_a = [&](int J, halfx8 (&ah)[CB], halfx8 (&al)[CB]) {
#pragma unroll
    for (int r = 0; r < CB; ++r) {
      const int blk = J * nrb + wave + 8 * r;
      ah[r] = __builtin_bit_cast(halfx8, ld4(g_rs, lane * 16, blk * 2048));
      al[r] = __builtin_bit_cast(halfx8, ld4(g_rs, lane * 16, blk * 2048 + 1024));
    }
  };

  floatx4 acc[CB][4];
#pragma unroll
  for (int r = 0; r < CB; ++r)
#pragma unroll
    for (int cb4 = 0; cb4 < 4; ++cb4) acc[r][cb4] = floatx4{0.f, 0.f, 0.f, 0.f};

  // prologue: blocks 0 and 1 produced, block 2's operands loaded
  prod_load(0);
  produce(0);
  if (a.n32 > 1) {
    prod_load(1);
    produce(1);
  }
  prod_load(2);
  halfx8 ah[CB], al[CB];
  load_a(0, ah, al);
  lds_sync();

  // One step: the MFMAs of block J (each product pass over all accumulators
  // before the next, so no MFMA waits on the one before it) and, when PROD,
  // the evaluation of block J + 2, interleaved by the scheduler pattern below;
  // then the operands of block J + 3.
  auto step = [&](int J, auto prod) {
    constexpr bool PROD = decltype(prod)::value;
    halfx8 bh[4], bl[4];
    const _Float16* kb = ring + (J % 3) * kRingSlot + (lane % 16) * kKS + 8 * (lane / 16);
#pragma unroll
    for (int cb4 = 0; cb4 < 4; ++cb4) {
      bh[cb4] = *reinterpret_cast<const halfx8*>(kb + 16 * cb4 * kKS);
      bl[cb4] = *reinterpret_cast<const halfx8*>(kb + 16 * cb4 * kKS + kPlane);
    }
    halfx8 nh[CB], nl[CB];
    load_a(min(J + 1, a.n32 - 1), nh, nl);
    if constexpr (PROD) produce(J + 2);
#pragma unroll
    for (int r = 0; r < CB; ++r)
#pragma unroll
      for (int cb4 = 0; cb4 < 4; ++cb4)
        acc[r][cb4] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[r], bh[cb4], acc[r][cb4], 0, 0, 0);
#pragma unroll
    for (int r = 0; r < CB; ++r)
#pragma unroll
      for (int cb4 = 0; cb4 < 4; ++cb4)
        acc[r][cb4] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[r], bl[cb4], acc[r][cb4], 0, 0, 0);
#pragma unroll
    for (int r = 0; r < CB; ++r)
#pragma unroll
      for (int cb4 = 0; cb4 < 4; ++cb4)
        acc[r][cb4] = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[r], bh[cb4], acc[r][cb4], 0, 0, 0);
    if constexpr (PROD) {
      // interleave the kernel-value VALU work with the MFMAs
      constexpr int nM = 12 * CB;
      constexpr int nV = 4 * (COMP ? 34 : 20);
#pragma unroll
      for (int i = 0; i < nM; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, (nV + nM - 1) / nM, 0);  // VALU
      }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int r = 0; r < CB; ++r) {
      ah[r] = nh[r];
      al[r] = nl[r];
    }
    if constexpr (PROD) prod_load(J + 3);
    lds_sync();
  };
  int J = 0;
  for (; J + 2 < a.n32; ++J) step(J, std::true_type{});
  for (; J < a.n32; ++J) step(J, std::false_type{});

  const float gi = a.ginv[k];
#pragma unroll
  for (int r = 0; r < CB; ++r)
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int64_t c = c0 + 16 * cb + lane % 16;
      const float sc = gi * kish[16 * cb + lane % 16];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int smp = 16 * (wave + 8 * r) + 4 * (lane / 16) + e;
        if (smp < a.S && c < a.npts) a.out[((int64_t)k * a.S + smp) * a.ldo + c] = acc[r][cb][e] * sc;
      }
    }
}

// ---- per-sample HVI -----------------------------------------------------------

// One lane per candidate batch. Draw s of member a, objective k:
//   y = mu_ak + D[k][s][b q + a] + (q = 1: tau_k z_s,k;
//                                   q > 1: sum_t C_k[a][t] z_s,t,k),
// then the HVI of the batch against the boxes of draw s (inclusion-exclusion
// over the member subsets for q > 1). All lanes are at the same draw, so the
// box loop is uniform and every box read is a broadcast: from LDS when the
// boxes fit there (LDSB), else from global memory. The constrained form
// replaces an infeasible member's first objective by -inf, which zeroes every
// term that contains it.
constexpr int kET = 512;   // threads per workgroup of the HVI kernel

template <int MO>
__device__ __forceinline__ float nz_mask(const float (&y)[MO], const NehviEhviArgs& a) {
  bool ok = true;
#pragma unroll
  for (int k = 0; k < MO; ++k) ok = ok && (y[k] >= a.low[k]);
  return ok ? y[0] : -__builtin_inff();
}

template <int MO, int Q, bool CONS, bool LDSB>
__global__ __launch_bounds__(kET) void k_nehvi_ehvi(NehviEhviArgs a) {
  extern __shared__ float esm[];
  constexpr int BW = 2 * MO;
  constexpr int T = Q * (Q + 1) / 2;
  constexpr int NS = 1 << Q;
  constexpr int U = (Q * MO <= 2) ? 16 : (Q * MO <= 4) ? 8 : (Q * MO <= 8) ? 4 : 2;
  float* zs = esm;                                                  // [S][Q][MO]
  int* off = reinterpret_cast<int*>(zs + a.S * Q * MO);            // [S + 1]
  float* bxl = reinterpret_cast<float*>(off + a.S + 1);            // [total][BW] (LDSB)
  for (int i = threadIdx.x; i < a.S * Q * MO; i += kET) zs[i] = a.Z[i];
  for (int i = threadIdx.x; i <= a.S; i += kET) off[i] = a.off[i];
  if constexpr (LDSB)
    for (int i = threadIdx.x; i < a.total * BW; i += kET) bxl[i] = a.boxes[i];
  __syncthreads();
  const float* bx = LDSB ? bxl : a.boxes;
  // q > 1: batches are few (65,536 per chunk at q = 4), so the waves of a
  // workgroup share 64 batches and split the draws; their partial sums are
  // added in LDS in wave order. q = 1: a lane per batch over all draws.
  constexpr bool SPLIT = Q > 1;
  constexpr int kEW = kET / 64;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t b = SPLIT ? (int64_t)blockIdx.x * 64 + lane : (int64_t)blockIdx.x * kET + threadIdx.x;
  int sbeg = 0, send = a.S;
  if constexpr (SPLIT) {
    const int sw = (a.S + kEW * U - 1) / (kEW * U) * U;
    sbeg = wave * sw;
    send = min(a.S, sbeg + sw);
  }
  const bool valid = b < a.nbat;
  const int64_t bb = valid ? b : a.nbat - 1;
  float mu[Q][MO];
  float C[MO][T];                       // q = 1: C[k][0] = tau_k
  bool nan_in = false;                  // a NaN posterior gives a NaN acquisition
#pragma unroll
  for (int i = 0; i < Q; ++i)
#pragma unroll
    for (int k = 0; k < MO; ++k) {
      mu[i][k] = a.mu[k * a.nbat * Q + bb * Q + i];
      nan_in = nan_in || (mu[i][k] != mu[i][k]);
    }
#pragma unroll
  for (int k = 0; k < MO; ++k)
#pragma unroll
    for (int e = 0; e < T; ++e) {
      C[k][e] = (Q == 1) ? a.sd[k * a.nbat + bb] : a.chol[(k * a.nbat + bb) * T + e];
      nan_in = nan_in || (C[k][e] != C[k][e]);
    }
  const float* dp = a.D + bb * Q;
  const int64_t kstride = (int64_t)a.S * a.ldd;
  float acc_pos = 0.f, acc_neg = 0.f;
  for (int s0 = sbeg; s0 < send; s0 += U) {
    float dv[U][Q][MO];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = min(s0 + u, send - 1);
#pragma unroll
      for (int k = 0; k < MO; ++k)
#pragma unroll
        for (int i = 0; i < Q; ++i) dv[u][i][k] = dp[k * kstride + (int64_t)s * a.ldd + i];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = s0 + u;
      if (s >= send) continue;    // uniform: the tail of the last group
      float y[Q][MO];
#pragma unroll
      for (int k = 0; k < MO; ++k)
#pragma unroll
        for (int i = 0; i < Q; ++i) {
          float v = mu[i][k] + dv[u][i][k];
#pragma unroll
          for (int t = 0; t <= i; ++t) v = fmaf(C[k][i * (i + 1) / 2 + t], zs[(s * Q + t) * MO + k], v);
          y[i][k] = v;
        }
      if constexpr (CONS) {
#pragma unroll
        for (int i = 0; i < Q; ++i) y[i][0] = nz_mask<MO>(y[i], a);
      }
      float ymax[MO];       // the batch's best value per objective in this draw
#pragma unroll
      for (int k = 0; k < MO; ++k) {
        float v = y[0][k];
#pragma unroll
        for (int i = 1; i < Q; ++i) v = fmaxf(v, y[i][k]);
        ymax[k] = v;
      }
      const int c0 = __builtin_amdgcn_readfirstlane(off[s]);
      const int c1 = __builtin_amdgcn_readfirstlane(off[s + 1]);
      for (int c = c0; c < c1; ++c) {
        float lo[MO], w[MO];
#pragma unroll
        for (int k = 0; k < MO; ++k) {
          lo[k] = bx[c * BW + k];
          w[k] = bx[c * BW + MO + k];
        }
        if constexpr (Q > 1 || MO > 2) {
          // a box whose lower corner no member exceeds in some objective adds
          // exactly zero; skip it when that holds on every lane
          bool nz = true;
#pragma unroll
          for (int k = 0; k < MO; ++k) nz = nz && (ymax[k] > lo[k]);
          if (__ballot(nz) == 0) continue;
        }
        if constexpr (Q > 1) {
          // the members that reach the box (above its lower corner in every
          // objective) on some lane: when only one does, the box adds that
          // member's own extent product (the other subset terms are zeros)
          int rmask = 0;
#pragma unroll
          for (int i = 0; i < Q; ++i) {
            bool r = true;
#pragma unroll
            for (int k = 0; k < MO; ++k) r = r && (y[i][k] > lo[k]);
            if (__ballot(r) != 0) rmask |= 1 << i;
          }
          if (rmask == 0) continue;
          if ((rmask & (rmask - 1)) == 0) {
#pragma unroll
            for (int i = 0; i < Q; ++i) {
              if (rmask == (1 << i)) {
                float t = __builtin_amdgcn_fmed3f(y[i][0] - lo[0], 0.f, w[0]);
#pragma unroll
                for (int k = 1; k < MO; ++k) t *= __builtin_amdgcn_fmed3f(y[i][k] - lo[k], 0.f, w[k]);
                acc_pos += t;
              }
            }
            continue;
          }
        }
        if constexpr (Q == 1) {
          float t = __builtin_amdgcn_fmed3f(y[0][0] - lo[0], 0.f, w[0]);
#pragma unroll
          for (int k = 1; k < MO; ++k) t *= __builtin_amdgcn_fmed3f(y[0][k] - lo[k], 0.f, w[k]);
          acc_pos += t;
        } else {
          float ext[NS][MO];
#pragma unroll
          for (int i = 0; i < Q; ++i)
#pragma unroll
            for (int k = 0; k < MO; ++k)
              ext[1 << i][k] = __builtin_amdgcn_fmed3f(y[i][k] - lo[k], 0.f, w[k]);
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
  }
  if constexpr (SPLIT) {
    __syncthreads();                    // the draws' LDS is done with
    float* part = esm;                  // [kEW][64]
    part[wave * 64 + lane] = acc_pos - acc_neg;
    __syncthreads();
    if (wave == 0) {
      float tot = 0.f;
#pragma unroll
      for (int w = 0; w < kEW; ++w) tot += part[w * 64 + lane];
      if (valid) a.ehvi[b] = nan_in ? __builtin_nanf("") : tot / static_cast<float>(a.S);
    }
  } else {
    if (valid) a.ehvi[b] = nan_in ? __builtin_nanf("") : (acc_pos - acc_neg) / static_cast<float>(a.S);
  }
}

template <int MO, int Q, bool CONS>
hipError_t nz_ehvi_launch(const NehviEhviArgs& a, bool ldsb, size_t lds, unsigned grid,
                          hipStream_t st) {
  // more than 64 KiB of dynamic LDS: opt in on every launch, so that it holds
  // on whichever device is current
  const void* f = ldsb ? reinterpret_cast<const void*>(&k_nehvi_ehvi<MO, Q, CONS, true>)
                       : reinterpret_cast<const void*>(&k_nehvi_ehvi<MO, Q, CONS, false>);
  hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  if (e != hipSuccess) return e;
  if (ldsb) hipLaunchKernelGGL((k_nehvi_ehvi<MO, Q, CONS, true>), dim3(grid), dim3(kET), lds, st, a);
  else hipLaunchKernelGGL((k_nehvi_ehvi<MO, Q, CONS, false>), dim3(grid), dim3(kET), lds, st, a);
  return hipGetLastError();
}

template <int MO, bool CONS>
hipError_t nz_ehvi_q(const NehviEhviArgs& a, bool ldsb, size_t lds, unsigned grid, hipStream_t st) {
  switch (a.q) {
    case 1: return nz_ehvi_launch<MO, 1, CONS>(a, ldsb, lds, grid, st);
    case 2: return nz_ehvi_launch<MO, 2, CONS>(a, ldsb, lds, grid, st);
    case 4: return nz_ehvi_launch<MO, 4, CONS>(a, ldsb, lds, grid, st);
  }
  return hipErrorInvalidValue;
}

template <int DX4, bool COMP>
hipError_t means_dx(const NehviMeansArgs& a, dim3 grid, hipStream_t st) {
  switch (a.S <= 128 ? 1 : a.S <= 256 ? 2 : a.S <= 384 ? 3 : 4) {
    case 1: hipLaunchKernelGGL((k_nehvi_means<DX4, 1, COMP>), grid, dim3(kMW * 64), 0, st, a); break;
    case 2: hipLaunchKernelGGL((k_nehvi_means<DX4, 2, COMP>), grid, dim3(kMW * 64), 0, st, a); break;
    case 3: hipLaunchKernelGGL((k_nehvi_means<DX4, 3, COMP>), grid, dim3(kMW * 64), 0, st, a); break;
    default: hipLaunchKernelGGL((k_nehvi_means<DX4, 4, COMP>), grid, dim3(kMW * 64), 0, st, a); break;
  }
  return hipGetLastError();
}

}  // namespace

size_t nehvi_front_lds_bytes(int64_t n) {
  return sizeof(double) * 2 * n + sizeof(int) * 3 * n;
}

size_t nehvi_ehvi_lds_bytes(int S, int q, int m, int total, bool boxes_in_lds) {
  return sizeof(float) * ((size_t)S * q * m + (boxes_in_lds ? 2 * (size_t)m * total : 0)) +
         sizeof(int) * ((size_t)S + 1);
}

int nehvi_padded_samples(int S) { return (S + 127) / 128 * 128; }

hipError_t launch_sample_fronts(const NehviFrontArgs& a, hipStream_t st) {
  // at most 28 n bytes (57 KiB at n = 2048): within the default limit
  const size_t lds = nehvi_front_lds_bytes(a.n);
  hipLaunchKernelGGL(k_sample_front, dim3(a.S), dim3(256), lds, st, a);
  return hipGetLastError();
}

size_t nehvi_front3_lds_bytes(int64_t n) {
  return sizeof(double) * 6 * n + sizeof(int) * 3 * n;
}

hipError_t launch_sample_fronts3(const NehviFront3Args& a, hipStream_t st) {
  // 60 n bytes (120 KiB at n = 2048): beyond the default dynamic limit
  const size_t lds = nehvi_front3_lds_bytes(a.n);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_sample_front3),
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     static_cast<int>(lds));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_sample_front3, dim3(a.S), dim3(256), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_compact_boxes3(const float* tmp, int64_t stride, const int* off, int S,
                                 float* out, hipStream_t st) {
  hipLaunchKernelGGL(k_compact_boxes3, dim3(S), dim3(64), 0, st, tmp, stride, off, out);
  return hipGetLastError();
}

hipError_t launch_absmax(const double* G, int64_t count, int m, double* part, hipStream_t st) {
  hipLaunchKernelGGL(k_absmax, dim3(kAbsmaxParts, m), dim3(256), 0, st, G, count, part);
  return hipGetLastError();
}

hipError_t launch_pack_g(const double* G, int nf, int Sp, int n32, int m, const float* scale,
                         uint16_t* Gp, hipStream_t st) {
  const int nrb = Sp / 16;
  const unsigned g = static_cast<unsigned>(((int64_t)n32 * nrb * 64 + 255) / 256);
  hipLaunchKernelGGL(k_pack_g, dim3(g, m), dim3(256), 0, st, G, nf, Sp, n32, nrb, scale[0],
                     m > 1 ? scale[1] : 1.f, m > 2 ? scale[2] : 1.f,
                     reinterpret_cast<_Float16*>(Gp));
  return hipGetLastError();
}

hipError_t launch_compact_boxes(const float* tmp, int64_t stride, const int* off, int S,
                                float* out, hipStream_t st) {
  hipLaunchKernelGGL(k_compact_boxes, dim3(S), dim3(64), 0, st, tmp, stride, off, out);
  return hipGetLastError();
}

hipError_t launch_nehvi_means(const NehviMeansArgs& a, int m, hipStream_t st) {
  if (a.npts <= 0) return hipSuccess;
  if (a.S < 1 || a.S > 512 || a.dx % 4 != 0 || a.dx > BO_MAX_D) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>((a.npts + kMT - 1) / kMT), m);
  if (a.dr > 0) {
    // a composite model has at least two coordinate groups
    switch (a.dx / 4) {
      case 2: return means_dx<2, true>(a, grid, st);
      case 3: return means_dx<3, true>(a, grid, st);
      case 4: return means_dx<4, true>(a, grid, st);
      case 5: return means_dx<5, true>(a, grid, st);
      case 6: return means_dx<6, true>(a, grid, st);
      case 7: return means_dx<7, true>(a, grid, st);
      case 8: return means_dx<8, true>(a, grid, st);
    }
    return hipErrorInvalidValue;
  }
  switch (a.dx / 4) {
    case 1: return means_dx<1, false>(a, grid, st);
    case 2: return means_dx<2, false>(a, grid, st);
    case 3: return means_dx<3, false>(a, grid, st);
    case 4: return means_dx<4, false>(a, grid, st);
    case 5: return means_dx<5, false>(a, grid, st);
    case 6: return means_dx<6, false>(a, grid, st);
    case 7: return means_dx<7, false>(a, grid, st);
    case 8: return means_dx<8, false>(a, grid, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_nehvi_ehvi(const NehviEhviArgs& a, hipStream_t st) {
  if (a.nbat <= 0) return hipSuccess;
  const bool ldsb = nehvi_ehvi_lds_bytes(a.S, a.q, a.m, a.total, true) <= 160 * 1024;
  // (q > 1: at least the waves' partial sums, which reuse the space at the end)
  const size_t lds = std::max<size_t>(nehvi_ehvi_lds_bytes(a.S, a.q, a.m, a.total, ldsb),
                                      a.q > 1 ? sizeof(float) * kET : 0);
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  // q = 1: a lane per batch; q > 1: a workgroup per 64 batches
  const int per = (a.q == 1) ? kET : 64;
  const unsigned grid = static_cast<unsigned>((a.nbat + per - 1) / per);
  if (a.m == 2) return a.cons ? nz_ehvi_q<2, true>(a, ldsb, lds, grid, st)
                              : nz_ehvi_q<2, false>(a, ldsb, lds, grid, st);
  if (a.m == 3) return a.cons ? nz_ehvi_q<3, true>(a, ldsb, lds, grid, st)
                              : nz_ehvi_q<3, false>(a, ldsb, lds, grid, st);
  return hipErrorInvalidValue;
}

hipError_t launch_insample_values(const float* Y, const double* alpha64, const double* noise,
                                  const double* T1, int64_t n, int m, int nf, int Sp, int S,
                                  double* F, hipStream_t st) {
  const unsigned g = static_cast<unsigned>(((int64_t)S * n + 255) / 256);
  hipLaunchKernelGGL(k_insample_values, dim3(g, m), dim3(256), 0, st, Y, alpha64, noise, T1, n, m,
                     nf, Sp, S, F);
  return hipGetLastError();
}

}  // namespace bo
