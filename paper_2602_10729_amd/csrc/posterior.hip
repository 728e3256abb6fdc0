// GP posterior of a batch of candidate points, one objective per launch.
//
// Paper: workflow step (ii) evaluates the acquisition on samples of the
// joint posterior of the GP surrogates; the posterior of an exact GP at x*
// is mu = k*^T alpha and Sigma = k(x*,x*) - v^T v with v = L^{-1} k*.
//
// One workgroup (8 waves, two per SIMD) owns a tile of NT points and forms
// V = L^{-1} K*^T left-looking: the outer loop runs over the 16-row blocks J
// of K*^T, and every wave adds L^{-1}[I][J] K*^T[J] into the accumulators of
// the row blocks I >= J that it owns. Row block I of V therefore never
// leaves the MFMA accumulators until it is complete, and then only its
// squared column sums (q = 1: |v|^2; q > 1 also the cross products of batch
// members, which sit in the same 4-lane group and are exchanged with DPP
// quad permutes) are kept.
//
// K*^T is never resident as a whole: it is produced on the fly, one block
// ahead of its use, into a two-chunk LDS ring (a chunk is 64 rows). While
// the matrix core works on block J, the same waves evaluate the ARD
// Matern-5/2 values of block J + 4 on the vector ALUs (direct differences
// of lengthscale-scaled coordinates, no |a|^2 + |b|^2 - 2ab cancellation)
// and accumulate mu = K* alpha. One barrier per chunk publishes it.
//
// Each wave owns RB row-block slots, slot r holding row block
// base + 8r + (r even ? wave : 7 - wave); this snake keeps the per-SIMD
// share of the lower triangle even at every step of J. Row blocks beyond
// the matrix (and finished slots) read a zero block appended to the packed
// L^{-1}, so every load is unconditional and in bounds. For n_pad > 128 RB
// rows the rows are handled in passes of 8 RB blocks, K*^T being produced
// again for each pass.
//
// The 16 inner indices of a block are split as k = 4g + kk between the four
// 16-lane groups g and the four MFMA steps kk, so each lane's four A
// operands are four consecutive columns of L^{-1} (pre-packed by the fit: one
// 16-byte load, 1 KiB per block per wave) and its four B operands are four
// consecutive rows of K*^T (one 16-byte LDS read).
// MFMA: v_mfma_f32_16x16x4f32, A[i][k] from lane i + 16k, B[k][j] from lane
// j + 16k, D[i][j] in lane j + 16(i/4), element i%4.
#include <hip/hip_runtime.h>

#include "bo_internal.h"

namespace bo {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

#ifndef BO_POST_NT
#define BO_POST_NT 32        // points per tile
#endif
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kChunkRows = 64;              // rows of K*^T per ring chunk
constexpr int kCS = kChunkRows + 4;         // column stride in the ring (mod 32 banks: 4)

__device__ inline float matern52_f(float r2, float s) {
  const float r = __builtin_amdgcn_sqrtf(r2);
  // exp(-sqrt5 r) = 2^(-sqrt5 log2(e) r)
  constexpr float kNegSqrt5Log2e = static_cast<float>(-2.23606797749978969641 * 1.44269504088896340736);
  const float e = __builtin_amdgcn_exp2f(kNegSqrt5Log2e * r);
  const float poly = fmaf(r, 2.23606798f, fmaf(r2, 1.66666667f, 1.0f));
  return s * poly * e;
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

// LDS-only barrier: waits for this wave's LDS traffic, not for its global
// loads in flight (the A-fragment prefetches), then joins the workgroup.
__device__ inline void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Per-lane state of the K*^T producer: this lane evaluates row (lane & 15)
// of each block for CPL columns of the tile.
template <int NT, int DX4>
struct Producer {
  static constexpr int CPL = NT / 32;
  float c[CPL][DX4 * 4];    // scaled candidate coordinates
  bool valid[CPL];
  float mu[CPL];
  float4 xn[DX4];           // training row of the next block
  float aln;                // alpha of that row
  int col0;                 // first tile column of this lane
  __amdgpu_buffer_rsrc_t xs_rs, al_rs;   // scaled X, alpha
};

// Raw buffer resource over `bytes` bytes at p: loads take a 32-bit lane
// offset plus a uniform offset, and read zero past the end.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}

__device__ __forceinline__ float4 load4(__amdgpu_buffer_rsrc_t rs, int voff, int soff) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, soff, 0));
}

template <int NT, int DX4>
__device__ __forceinline__ void producer_fetch(Producer<NT, DX4>& P, const PosteriorArgs& a,
                                               int n_pad, int jb, int rr) {
  const int row = min(jb * kBlk + rr, n_pad - 1);
#pragma unroll
  for (int t4 = 0; t4 < DX4; ++t4) P.xn[t4] = load4(P.xs_rs, (row * a.dx + 4 * t4) * 4, 0);
  P.aln = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(P.al_rs, row * 4, 0, 0));
}

// Evaluate block jb of K*^T (the one fetched last) into the ring, then fetch
// block jb + 1. Blocks past the matrix produce zeros that are never read.
template <int NT, int DX4>
__device__ __forceinline__ void produce(Producer<NT, DX4>& P, const PosteriorArgs& a, int n_pad,
                                        int jb, int rr, float* ring) {
  constexpr int CPL = NT / 32;
  const int row = jb * kBlk + rr;
  const bool live = row < a.n;
  float* dst = ring + ((jb >> 2) & 1) * (NT * kCS) + (jb & 3) * kBlk + rr;
#pragma unroll
  for (int u = 0; u < CPL; ++u) {
    float r2 = 0.f;
#pragma unroll
    for (int t4 = 0; t4 < DX4; ++t4) {
      const float d0 = P.c[u][4 * t4 + 0] - P.xn[t4].x;
      const float d1 = P.c[u][4 * t4 + 1] - P.xn[t4].y;
      const float d2 = P.c[u][4 * t4 + 2] - P.xn[t4].z;
      const float d3 = P.c[u][4 * t4 + 3] - P.xn[t4].w;
      r2 = fmaf(d0, d0, r2);
      r2 = fmaf(d1, d1, r2);
      r2 = fmaf(d2, d2, r2);
      r2 = fmaf(d3, d3, r2);
    }
    const float kv = (P.valid[u] && live) ? matern52_f(r2, a.s) : 0.f;
    P.mu[u] = fmaf(P.aln, kv, P.mu[u]);
    dst[(P.col0 + u) * kCS] = kv;
  }
  producer_fetch(P, a, n_pad, jb + 1, rr);
}

// Row block of slot r in the pass starting at row block `base`.
__device__ inline int slot_block(int base, int r, int wave) {
  return base + 8 * r + ((r & 1) ? (kWaves - 1 - wave) : wave);
}

// Row-block slots of a wave in one pass: fragment index of block (I, 0) and
// I itself, or (zero block, -1) for a slot past the matrix. Block (I, J) of
// a slot is first + J while J <= I, the zero block afterwards.
template <int RB>
struct Slots {
  int first[RB];
  int last[RB];
};

__device__ __forceinline__ int frag_block(int first, int last, int J, int zero_blk) {
  return (J <= last) ? first + J : zero_blk;
}

// MFMAs of one K*^T block for the slots [LO, RB), taken two slots at a time
// (four independent accumulators per inner step); each pair's fragments for
// the next block are requested as soon as its MFMAs are issued, so they
// have a whole step to arrive.
template <int LO, int RB, int NCB>
__device__ __forceinline__ void mfma_slots(float4 (&av)[RB], const float4 (&bv)[NCB],
                                           floatx4 (&acc)[RB][NCB], __amdgpu_buffer_rsrc_t lp_rs,
                                           const Slots<RB>& sl, int Jn, int zero_blk, int voff) {
#pragma unroll
  for (int r0 = LO; r0 < RB; r0 += 2) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int r = r0; r < r0 + 2 && r < RB; ++r)
#pragma unroll
        for (int b = 0; b < NCB; ++b) {
          const float A = kk == 0 ? av[r].x : kk == 1 ? av[r].y : kk == 2 ? av[r].z : av[r].w;
          const float B = kk == 0 ? bv[b].x : kk == 1 ? bv[b].y : kk == 2 ? bv[b].z : bv[b].w;
          acc[r][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(A, B, acc[r][b], 0, 0, 0);
        }
#pragma unroll
    for (int r = r0; r < r0 + 2 && r < RB; ++r)
      av[r] = load4(lp_rs, voff, frag_block(sl.first[r], sl.last[r], Jn, zero_blk) * 1024);
  }
}

// Workgroup-uniform context of the streaming loop.
struct Ctx {
  __amdgpu_buffer_rsrc_t lp_rs;   // packed fragments of this objective
  int nb, zero_blk, n_pad, wave, rr;
  int voff;            // this lane's byte offset inside a fragment block
  const float* Kb;     // this lane's B-fragment base inside the ring
};

// One step J for slots [LO, RB): B fragments of block J, the producer's
// block J + 4, the MFMAs with the slots' fragments for J + 1, and the chunk
// barrier after the last block of a chunk.
template <int LO, int RB, int NT, int DX4>
__device__ __forceinline__ void step(const Ctx& C, const PosteriorArgs& a, Producer<NT, DX4>& P,
                                     float* ring, const Slots<RB>& sl, int J, float4 (&av)[RB],
                                     floatx4 (&acc)[RB][NT / 16]) {
  constexpr int NCB = NT / 16;
  float4 bv[NCB];
  const float* kb = C.Kb + ((J >> 2) & 1) * (NT * kCS) + (J & 3) * kBlk;
#pragma unroll
  for (int b = 0; b < NCB; ++b) bv[b] = *reinterpret_cast<const float4*>(kb + b * 16 * kCS);
  produce(P, a, C.n_pad, J + 4, C.rr, ring);
  mfma_slots<LO, RB, NCB>(av, bv, acc, C.lp_rs, sl, J + 1, C.zero_blk, C.voff);
  if ((J & 3) == 3) lds_barrier();
}

// Rounds R.. of the triangular part of a pass: in round R (blocks
// J in [base + 8R, base + 8R + 8)) slot R is live while J <= its row block,
// slots above R throughout.
template <int R, int RB, int NT, int DX4>
__device__ __forceinline__ void rounds(const Ctx& C, const PosteriorArgs& a, Producer<NT, DX4>& P,
                                       float* ring, const Slots<RB>& sl, int base,
                                       float4 (&av)[RB], floatx4 (&acc)[RB][NT / 16]) {
  if constexpr (R < RB) {
    const int j0 = base + 8 * R;
    if (j0 >= C.nb) return;
    const int jend = min(j0 + 8, C.nb);
    const int jlive = min(slot_block(base, R, C.wave) + 1, jend);
    int J = j0;
    for (; J < jlive; ++J) step<R, RB, NT, DX4>(C, a, P, ring, sl, J, av, acc);
    for (; J < jend; ++J) step<R + 1, RB, NT, DX4>(C, a, P, ring, sl, J, av, acc);
    rounds<R + 1, RB, NT, DX4>(C, a, P, ring, sl, base, av, acc);
  }
}

template <int NT, int DX4, int Q, int RB>
__global__ __launch_bounds__(kThreads) void k_posterior(PosteriorArgs a) {
  extern __shared__ float smem[];
  constexpr int NCB = NT / 16;          // 16-column blocks per tile
  constexpr int NX = (Q > 1) ? Q : 1;   // per-point partial slots (diag + xors)
  constexpr int CPL = NT / 32;
  static_assert(NT == 32 || NT == 64, "tile width");
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // wave index as a scalar: the loop control below stays uniform
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n_pad = a.nb * kBlk;
  float* ring = smem;                                // 2 chunks x NT x kCS
  float* red = ring + 2 * NT * kCS;                  // kWaves * NT * NX
  float* mush = red + kWaves * NT * NX;              // NT
  float* kpp = mush + NT;                            // NT * 4 (prior cross-cov)
  const int64_t p0 = (int64_t)blockIdx.x * NT;
  const int rr = lane & 15;

  Producer<NT, DX4> P;
  P.col0 = wave * (NT / 8) + (lane >> 4) * CPL;
#pragma unroll
  for (int u = 0; u < CPL; ++u) {
    const int64_t p = p0 + P.col0 + u;
    P.valid[u] = p < a.npts;
#pragma unroll
    for (int t = 0; t < DX4 * 4; ++t) P.c[u][t] = 0.f;
    if (P.valid[u]) {
      const float* cp = a.cand + p * a.d;
#pragma unroll
      for (int t = 0; t < DX4 * 4; ++t)
        if (t < a.d) P.c[u][t] = cp[t] * a.invls[t];
    }
  }

  if (Q > 1) {
    // prior covariance of each point with its batch mates (point ^ x),
    // partner x on lane rr = x of the column's 16-lane group
#pragma unroll
    for (int u = 0; u < CPL; ++u) {
      const int colu = P.col0 + u;
      if (rr >= 1 && rr < Q) {
        const int64_t pm = (p0 + colu) ^ rr;
        float r2 = 0.f;
        if (P.valid[u] && pm < a.npts) {
          const float* cp = a.cand + pm * a.d;
#pragma unroll
          for (int t = 0; t < DX4 * 4; ++t)
            if (t < a.d) {
              const float dd = P.c[u][t] - cp[t] * a.invls[t];
              r2 = fmaf(dd, dd, r2);
            }
        }
        kpp[colu * 4 + rr] = matern52_f(r2, a.s);
      }
    }
  }

  Ctx C;
  C.nb = a.nb;
  C.zero_blk = a.nb * (a.nb + 1) / 2;
  C.lp_rs = make_rsrc(a.Lp, (C.zero_blk + 1) * 1024);
  P.xs_rs = make_rsrc(a.Xs, n_pad * a.dx * 4);
  P.al_rs = make_rsrc(a.alpha, n_pad * 4);
  C.n_pad = n_pad;
  C.wave = wave;
  C.rr = rr;
  C.voff = lane * 16;
  // B fragments: column (b*16 + lane%16), rows 4*(lane/16) .. +3 of a block
  C.Kb = ring + (size_t)(lane & 15) * kCS + 4 * (lane >> 4);

  float ss[NCB];
  float gx[NCB][NX];
#pragma unroll
  for (int b = 0; b < NCB; ++b) {
    ss[b] = 0.f;
#pragma unroll
    for (int x = 0; x < NX; ++x) gx[b][x] = 0.f;
  }

  for (int base = 0; base < a.nb; base += 8 * RB) {
    floatx4 acc[RB][NCB];
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
      for (int b = 0; b < NCB; ++b) acc[r][b] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < CPL; ++u) P.mu[u] = 0.f;
    Slots<RB> sl;
    float4 av[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int I = slot_block(base, r, wave);
      sl.first[r] = I < a.nb ? I * (I + 1) / 2 : C.zero_blk;
      sl.last[r] = I < a.nb ? I : -1;
      av[r] = load4(C.lp_rs, C.voff, frag_block(sl.first[r], sl.last[r], 0, C.zero_blk) * 1024);
    }
    // the previous pass may still read chunk 0 of the ring
    lds_barrier();
    producer_fetch(P, a, n_pad, 0, rr);
#pragma unroll
    for (int jb = 0; jb < 4; ++jb) produce(P, a, n_pad, jb, rr, ring);
    lds_barrier();
    // blocks left of this pass's triangle: every slot is live
    for (int J = 0; J < base; ++J) step<0, RB, NT, DX4>(C, a, P, ring, sl, J, av, acc);
    rounds<0, RB, NT, DX4>(C, a, P, ring, sl, base, av, acc);

#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
      for (int b = 0; b < NCB; ++b)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float v = acc[r][b][e];
          ss[b] = fmaf(v, v, ss[b]);
          if (Q > 1) {
#pragma unroll
            for (int x = 1; x < NX; ++x) gx[b][x] = fmaf(v, quad_xor(v, x), gx[b][x]);
          }
        }
  }

  // mu: the last pass produced every block; reduce over the 16 lanes of a
  // column
#pragma unroll
  for (int u = 0; u < CPL; ++u) {
    float v = P.mu[u];
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if (rr == 0) mush[P.col0 + u] = v;
  }
  // |v|^2 (and cross terms): over the four 16-lane row groups, then over
  // waves in LDS
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
        float L[Q][Q];
#pragma unroll
        for (int i = 0; i < Q; ++i)
#pragma unroll
          for (int j = 0; j < Q; ++j) L[i][j] = 0.f;
        const float tol = 1e-10f * a.s;
#pragma unroll
        for (int j = 0; j < Q; ++j) {
          float pv = S[j][j];
#pragma unroll
          for (int t = 0; t < j; ++t) pv = fmaf(-L[j][t], L[j][t], pv);
          if (pv > tol) {
            const float ljj = __builtin_amdgcn_sqrtf(pv);
            L[j][j] = ljj;
            const float inv = 1.0f / ljj;
#pragma unroll
            for (int i = j + 1; i < Q; ++i) {
              float num = S[i][j];
#pragma unroll
              for (int t = 0; t < j; ++t) num = fmaf(-L[i][t], L[j][t], num);
              L[i][j] = num * inv;
            }
          }
        }
        constexpr int T = Q * (Q + 1) / 2;
        float* dst = a.chol + (bat * a.m + a.k) * T;
#pragma unroll
        for (int i = 0; i < Q; ++i)
#pragma unroll
          for (int j = 0; j <= i; ++j) dst[i * (i + 1) / 2 + j] = L[i][j];
      }
    }
  }
}

constexpr size_t lds_floats(int NT, int q) {
  return (size_t)2 * NT * kCS + (size_t)kWaves * NT * ((q > 1) ? q : 1) + NT + (size_t)NT * 4;
}

template <int NT, int DX4, int Q, int RB>
hipError_t launch_t(const PosteriorArgs& a, hipStream_t st) {
  const size_t lds = sizeof(float) * lds_floats(NT, Q);
  const unsigned grid = static_cast<unsigned>((a.npts + NT - 1) / NT);
  hipLaunchKernelGGL((k_posterior<NT, DX4, Q, RB>), dim3(grid), dim3(kThreads), lds, st, a);
  return hipGetLastError();
}

template <int NT, int Q, int RB>
hipError_t launch_dx(const PosteriorArgs& a, hipStream_t st) {
  switch (a.dx / 4) {
    case 1: return launch_t<NT, 1, Q, RB>(a, st);
    case 2: return launch_t<NT, 2, Q, RB>(a, st);
    case 3: return launch_t<NT, 3, Q, RB>(a, st);
    case 4: return launch_t<NT, 4, Q, RB>(a, st);
    case 5: return launch_t<NT, 5, Q, RB>(a, st);
    case 6: return launch_t<NT, 6, Q, RB>(a, st);
    case 7: return launch_t<NT, 7, Q, RB>(a, st);
    case 8: return launch_t<NT, 8, Q, RB>(a, st);
    default: return hipErrorInvalidValue;
  }
}

template <int NT, int RB>
hipError_t launch_q(const PosteriorArgs& a, hipStream_t st) {
  switch (a.q) {
    case 1: return launch_dx<NT, 1, RB>(a, st);
    case 2: return launch_dx<NT, 2, RB>(a, st);
    case 4: return launch_dx<NT, 4, RB>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

size_t posterior_lds_bytes(int nb, int q) {
  (void)nb;
  return sizeof(float) * lds_floats(BO_POST_NT, q);
}

hipError_t launch_posterior(const PosteriorArgs& a, hipStream_t st) {
  if (a.npts <= 0) return hipSuccess;
  // row-block slots per wave: the smallest of 2, 4, 8 covering nb / 8
  if (a.nb <= 16) return launch_q<BO_POST_NT, 2>(a, st);
  if (a.nb <= 32) return launch_q<BO_POST_NT, 4>(a, st);
  return launch_q<BO_POST_NT, 8>(a, st);
}

}  // namespace bo
