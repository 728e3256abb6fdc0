// Posterior kernel templates, included by the per-coordinate-width
// translation units posterior_dx<N>.hip (each instantiates one width, so
// the build compiles them in parallel) and by posterior.hip (shared helpers).
//
#pragma once
// GP posterior of a batch of candidate points, one objective per launch.
//
// Paper: workflow step (ii) evaluates the acquisition on samples of the
// joint posterior of the GP surrogates; the posterior of an exact GP at x*
// is mu = k*^T alpha and Sigma = k(x*,x*) - v^T v with v = L^{-1} k*.
//
// Arithmetic. V = L^{-1} K*^T runs on the fp16 matrix cores with each
// operand split into two fp16 halves, x = x_hi + x_lo (x_hi = fp16(x),
// x_lo = fp16(x - x_hi)), and three products per pair,
//   a b ~ a_hi b_hi + a_hi b_lo + a_lo b_hi,
// accumulated in fp32 by the MFMA. Before the split both operands are scaled
// by powers of two: each 16-row block of L^{-1} so that its largest entry
// lies in [2^13, 2^14) (the fit does this once), each candidate's kernel
// values by 2^(14 - E), 2^E above a bound on its covariances (kv_split_scale).
// Nothing can then overflow fp16, and every entry within 2^-17 of its block's
// (or column's) largest has normal halves and 22 significant bits
// (|x - x_hi - x_lo| <= 2^-22 |x|); smaller entries carry an absolute error of
// at most 2^-39 of that largest. With the dropped a_lo b_lo term (2^-22
// relative) each product is within a few units of 2^-22 of exact, against
// 2^-23 for fp32 operands, and the products accumulate in fp32 as an fp32
// implementation's would. The scales are undone exactly: the row block's when
// a block of V is squared, the column's in the epilogue. On gfx950 this is
// the fast path: the dense fp16 MFMA runs at 16x the fp32 MFMA rate, and
// (unlike fp32 MFMA) it overlaps VALU work in part (each 16x16x32 MFMA takes
// about 8 cycles of its SIMD's VALU issue), which partly hides the kernel
// evaluations below. L^{-1} is split and packed once by the fit; K*^T is
// split as it is made.
//
// One workgroup (8 waves, two per SIMD) owns a tile of NT points and forms V
// left-looking: the outer loop runs over 32-row blocks J of K*^T (the MFMA
// k), and every wave adds L^{-1}[I][J] K*^T[J] into the accumulators of the
// 16-row blocks I >= 2J that it owns. Row block I of V stays in the MFMA
// accumulators until it is complete; then only its squared column sums
// (q = 1: |v|^2; q > 1 also the cross products of batch members, which sit
// in the same 4-lane group and are exchanged with DPP quad permutes) are
// kept.
//
// K*^T is produced two blocks ahead of its use into an LDS ring of 16
// blocks (512 rows) of fp16 hi/lo planes, from the training rows' distance
// fragments, norms and alpha, which each lane loads one step ahead into
// registers. While the matrix cores work on block J, the waves form the
// squared distances of block J + 2 with a few more MFMAs (the expansion
// |c|^2 + |x|^2 - 2c.x over centred coordinates, exact differences for pairs
// near a training point, see Producer), evaluate the ARD Matern-5/2 values on
// the vector ALUs and accumulate mu = K* alpha in fp32.
// A pass that starts while the ring still holds blocks 0.. reuses them, so
// for n <= 1024 every kernel value is evaluated once.
// The kernel evaluations and the MFMAs of a step are independent and are
// interleaved, so each SIMD's matrix core and vector ALU work together as far
// as their shared issue allows.
// One barrier per step publishes the produced block.
//
// Each wave owns RB row-block slots, slot r holding row block
// base + 8r + (r even ? wave : 7 - wave); this snake keeps the per-SIMD
// share of the lower triangle even at every step of J. Row blocks past the
// matrix (and finished slots) read a zero block appended to the packed
// L^{-1}, so every load is unconditional and in bounds. Rows beyond 128 RB
// are handled in further passes, K*^T being produced again for each pass
// (RB = 4: two passes for n = 1024; the accumulators of more rows would not
// fit the register file next to the operands).
//
// Fragments of v_mfma_f32_16x16x32_f16: A[i][k] from lane i + 16(k/8),
// element k%8; B[k][j] from lane j + 16(k/8), element k%8; D[i][j] in lane
// j + 16(i/4), element i%4. Only the pairing of A's and B's k matters, and
// both sides use this one.
#include <hip/hip_runtime.h>

#include "bo_internal.h"
#include "kv_scale.h"

namespace bo {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));

#ifndef BO_POST_NT
#define BO_POST_NT 64        // points per tile
#endif
#ifndef BO_POST_RB
#define BO_POST_RB 4         // row-block slots per wave (rows per pass / 128)
#endif
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kJ = 32;                      // rows of K*^T per step (MFMA k)
constexpr int kRing = 16;                   // K*^T blocks held in LDS
constexpr int kCSH = kRing * kJ + 8;        // ring column stride in halves (260 dwords)

__device__ __forceinline__ float matern52_f(float r2, float s) {
  const float r = __builtin_amdgcn_sqrtf(r2);
  // exp(-sqrt5 r) = 2^(-sqrt5 log2(e) r)
  constexpr float kNegSqrt5Log2e = static_cast<float>(-2.23606797749978969641 * 1.44269504088896340736);
  const float e = __builtin_amdgcn_exp2f(kNegSqrt5Log2e * r);
  const float poly = fmaf(r, 2.23606798f, fmaf(r2, 1.66666667f, 1.0f));
  return s * poly * e;
}

// Matern-3/2 correlation of squared scaled distance r2:
// (1 + sqrt3 r) exp(-sqrt3 r).
__device__ __forceinline__ float matern32_f(float r2) {
  const float r = __builtin_amdgcn_sqrtf(r2);
  constexpr float kNegSqrt3Log2e = static_cast<float>(-1.73205080756887729353 * 1.44269504088896340736);
  return fmaf(r, 1.73205081f, 1.0f) * __builtin_amdgcn_exp2f(kNegSqrt3Log2e * r);
}

__device__ __forceinline__ float quad_xor(float v, int x) {
  // DPP quad_perm: lane i of each group of 4 reads lane i ^ x.
  int iv = __float_as_int(v);
  int r;
  if (x == 1) r = __builtin_amdgcn_mov_dpp(iv, 0xB1, 0xF, 0xF, false);      // [1,0,3,2]
  else if (x == 2) r = __builtin_amdgcn_mov_dpp(iv, 0x4E, 0xF, 0xF, false); // [2,3,0,1]
  else r = __builtin_amdgcn_mov_dpp(iv, 0x1B, 0xF, 0xF, false);             // [3,2,1,0]
  return __int_as_float(r);
}

// LDS-only barrier: waits for this wave's LDS traffic, not for its global
// loads in flight (the fragment prefetches), then joins the workgroup.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Raw buffer resource over `bytes` bytes at p: loads take a 32-bit lane
// offset plus a uniform offset, and read zero past the end.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}

__device__ __forceinline__ float4 load4(__amdgpu_buffer_rsrc_t rs, int voff, int soff) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, soff, 0));
}

// Index of packed block (I, 0): row block I holds I/2 + 1 blocks of 32
// columns, so rows 0..I-1 hold t(t+1) (I = 2t) or (t+1)^2 (I = 2t+1).
__host__ __device__ __forceinline__ int frag_row_start(int I) {
  const int t = I >> 1;
  return (I & 1) ? (t + 1) * (t + 1) : t * (t + 1);
}

typedef _Float16 halfx4 __attribute__((ext_vector_type(4)));

// Per-lane state of the K*^T producer. Wave w makes rows 16(w/4) .. +15 and
// columns 16(w%4) .. +15 of every 32-row block, in the MFMA result layout:
// lane l holds column 16(w%4) + l%16 and rows 16(w/4) + 4(l/16) .. +3.
//
// Squared distances: r^2 = |c|^2 + |x|^2 - 2 c.x over coordinates centred on
// the training mean, c.x on the matrix cores from fp16 hi and 2^11-scaled lo
// halves (the fit packs the rows, the kernel the candidates; two accumulator
// streams, see dist_frags). Where the expansion can cancel badly, i.e. for a
// pair whose approximate r^2 is below 1 + (|c|^2 + |x|^2)/256, the pair is
// recomputed from exact differences of the scaled coordinates: near a
// training point k(x*, x_i) is close to its maximum and sigma^2 cancels,
// elsewhere the expansion's error (about 2^-20 (|c|^2 + |x|^2)) changes sigma
// by far less than its fp32 rounding. The choice is made per pair, so a
// point's result does not depend on its neighbours in the tile.
// Composite kernel: one expansion per coordinate group (routing slots first,
// then deployment), the candidate fragments masked to the group; the test
// above uses the total over both groups.
template <int NT, int DX4, bool COMP>
struct Producer {
  static constexpr int D = 4 * DX4;
  static constexpr int F0 = dist_frags0(D);
  static constexpr int NF = dist_frags(D);
  static constexpr int NS = COMP ? 2 : 1;
  static_assert(F0 == 1 && NF <= 3, "at most 32 coordinate slots");
  halfx8 cb[NS][NF];        // B fragments of this lane's candidate, per group
  float c2[NS];             // squared norm of the centred candidate, per group
  float mu;                 // sum of alpha times the scaled kernel values
  // composite: s_dep w(candidate), s_route and s_int, each times this column's
  // power-of-two split scale (a plain model's scaled s is uniform: a.ss)
  float wsd, ss, sis;
  int col;                  // tile column of this lane
  int rq;                   // first of this lane's rows inside a block
  int half;                 // row half of this wave
  // operands of the block made at the next step, loaded a step ahead
  halfx8 xa[NF];
  floatx4 x2[NS], al, wt;
  __amdgpu_buffer_rsrc_t xf_rs, x2_rs, al_rs, wt_rs, xs_rs;
};

// Load the operands of block jb (rows past the packed arrays read zero).
template <int NT, int DX4, bool COMP>
__device__ __forceinline__ void prod_load(Producer<NT, DX4, COMP>& P, int n_pad, int jb, int lane) {
  using Pr = Producer<NT, DX4, COMP>;
  const int vo = (2 * jb + P.half) * (Pr::NF * 1024) + lane * 16;
#pragma unroll
  for (int f = 0; f < Pr::NF; ++f)
    P.xa[f] = __builtin_bit_cast(halfx8, load4(P.xf_rs, vo + f * 1024, 0));
  const int row = jb * kJ + P.rq;
#pragma unroll
  for (int g = 0; g < Pr::NS; ++g)
    P.x2[g] = __builtin_bit_cast(floatx4, load4(P.x2_rs, ((COMP ? g : 1) * n_pad + row) * 4, 0));
  P.al = __builtin_bit_cast(floatx4, load4(P.al_rs, row * 4, 0));
  if constexpr (COMP) P.wt = __builtin_bit_cast(floatx4, load4(P.wt_rs, row * 4, 0));
}

// Squared scaled distances of this lane's four rows of block jb (operands
// loaded by prod_load). ctile: the tile's exact scaled candidate coordinates
// [NT][D]. Reads the operands' distance part only (xa, x2).
template <int NT, int DX4, bool COMP>
__device__ __forceinline__ void produce_dist(Producer<NT, DX4, COMP>& P, const PosteriorArgs& a, int jb,
                                             const float* ctile, float (&r2)[Producer<NT, DX4, COMP>::NS][4]) {
  using Pr = Producer<NT, DX4, COMP>;
  constexpr int NS = Pr::NS, F0 = Pr::F0, NF = Pr::NF;
  floatx4 d0[NS], d1[NS];
#pragma unroll
  for (int g = 0; g < NS; ++g) {
    d0[g] = floatx4{0.f, 0.f, 0.f, 0.f};
    d1[g] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int f = 0; f < F0; ++f)
      d0[g] = __builtin_amdgcn_mfma_f32_16x16x32_f16(P.xa[f], P.cb[g][f], d0[g], 0, 0, 0);
#pragma unroll
    for (int f = F0; f < NF; ++f)
      d1[g] = __builtin_amdgcn_mfma_f32_16x16x32_f16(P.xa[f], P.cb[g][f], d1[g], 0, 0, 0);
  }
  bool ex[4];
  bool any = false;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float rt = 0.f, nt = 0.f;
#pragma unroll
    for (int g = 0; g < NS; ++g) {
      const float nrm = P.c2[g] + P.x2[g][e];
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
    // zero coordinates)
    const float* cx = ctile + P.col * Pr::D;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = jb * kJ + P.rq + e;
      float s0 = 0.f, s1 = 0.f;   // routing / deployment (plain: s1 only)
#pragma unroll
      for (int t4 = 0; t4 < DX4; ++t4) {
        const float4 x = load4(P.xs_rs, (row * a.dx + 4 * t4) * 4, 0);
        const float4 c = *reinterpret_cast<const float4*>(cx + 4 * t4);
        const float e0 = c.x - x.x, e1 = c.y - x.y, e2 = c.z - x.z, e3 = c.w - x.w;
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
}

// Kernel values of this lane's four rows of block jb from their squared
// distances, alpha and (composite) weights, into the ring as fp16 hi/lo
// planes; adds them into mu.
template <int NT, int DX4, bool COMP>
__device__ __forceinline__ void produce_kv(Producer<NT, DX4, COMP>& P, const PosteriorArgs& a, int jb,
                                           const float (&r2)[Producer<NT, DX4, COMP>::NS][4],
                                           const floatx4& al, const floatx4& wt, _Float16* ring) {
  halfx4 hi, lo;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    // no mask: rows past n meet zero columns of L^{-1} and zero alpha;
    // columns past the batch are never written
    // the kernel value times this column's power-of-two split scale (the
    // scale rides in the output scales, so the product is exact)
    float kv;
    if constexpr (COMP) {
      // s_route M52(r_route) + s_dep w* w_i M32(r_dep) + s_int M52 M32
      const float k5 = matern52_f(r2[0][e], 1.0f);
      const float k3 = matern32_f(r2[1][e]);
      kv = fmaf(P.wsd * wt[e], k3, k5 * fmaf(P.sis, k3, P.ss));
    } else {
      kv = matern52_f(r2[0][e], a.ss);
    }
    // kv is rounded to fp32 here, once: otherwise the compiler may fuse its
    // last product into the fp16 conversions and derive the high half twice
    // (once exactly, once from the fp32 value); within an fp32 ulp of an
    // fp16 rounding midpoint the stored high and low halves then disagree by
    // one fp16 ulp. (The asm has no side effects: a volatile one would also
    // pin the loads and LDS accesses around it.)
    asm("" : "+v"(kv));
    P.mu = fmaf(al[e], kv, P.mu);
    const _Float16 h = static_cast<_Float16>(kv);
    hi[e] = h;
    lo[e] = static_cast<_Float16>(kv - static_cast<float>(h));
  }
  _Float16* dst = ring + P.col * kCSH + (jb % kRing) * kJ + P.rq;
  *reinterpret_cast<halfx4*>(dst) = hi;
  *reinterpret_cast<halfx4*>(dst + NT * kCSH) = lo;
}

// Both parts at once (operands loaded by prod_load).
template <int NT, int DX4, bool COMP>
__device__ __forceinline__ void produce(Producer<NT, DX4, COMP>& P, const PosteriorArgs& a, int jb,
                                        const float* ctile, _Float16* ring) {
  float r2[Producer<NT, DX4, COMP>::NS][4];
  produce_dist(P, a, jb, ctile, r2);
  produce_kv(P, a, jb, r2, P.al, P.wt, ring);
}

// Row block of slot r in the pass starting at row block `base`.
__device__ __forceinline__ int slot_block(int base, int r, int wave) {
  return base + 8 * r + ((r & 1) ? (kWaves - 1 - wave) : wave);
}

// Row-block slots of a wave in one pass: packed index of block (I, 0) and the
// last live J (I / 2), or (zero block, -1) for a slot past the matrix.
template <int RB>
struct Slots {
  int first[RB];
  int last[RB];
};

__device__ __forceinline__ int frag_block(int first, int last, int J, int zero_blk) {
  return (J <= last) ? first + J : zero_blk;
}

// A fragments of one slot: hi and lo planes (1 KiB each per block).
struct AFrag {
  halfx8 hi, lo;
};

__device__ __forceinline__ AFrag load_a(__amdgpu_buffer_rsrc_t rs, int voff, int blk) {
  AFrag f;
  f.hi = __builtin_bit_cast(halfx8, load4(rs, voff, blk * 2048));
  f.lo = __builtin_bit_cast(halfx8, load4(rs, voff, blk * 2048 + 1024));
  return f;
}

// B fragments of one half of a block (column blocks 2h and 2h + 1), hi and lo
// planes.
struct BHalf {
  halfx8 hi[2], lo[2];
};

// MFMAs of slots r0, r0 + 1 (those below RB) against one half of a block's
// columns: the three products of the pair's (up to) four accumulators.
template <int RB, int NCB, int H>
__device__ __forceinline__ void mfma_pair_half(int r0, const AFrag (&av)[RB], const BHalf& B,
                                               floatx4 (&acc)[RB][NCB]) {
#pragma unroll
  for (int r = r0; r < r0 + 2 && r < RB; ++r)
#pragma unroll
    for (int b = 0; b < 2; ++b)
      acc[r][2 * H + b] =
          __builtin_amdgcn_mfma_f32_16x16x32_f16(av[r].hi, B.hi[b], acc[r][2 * H + b], 0, 0, 0);
#pragma unroll
  for (int r = r0; r < r0 + 2 && r < RB; ++r)
#pragma unroll
    for (int b = 0; b < 2; ++b)
      acc[r][2 * H + b] =
          __builtin_amdgcn_mfma_f32_16x16x32_f16(av[r].hi, B.lo[b], acc[r][2 * H + b], 0, 0, 0);
#pragma unroll
  for (int r = r0; r < r0 + 2 && r < RB; ++r)
#pragma unroll
    for (int b = 0; b < 2; ++b)
      acc[r][2 * H + b] =
          __builtin_amdgcn_mfma_f32_16x16x32_f16(av[r].lo, B.hi[b], acc[r][2 * H + b], 0, 0, 0);
}

// Workgroup-uniform context of the streaming loop.
struct Ctx {
  __amdgpu_buffer_rsrc_t lp_rs;   // packed fragments of this objective
  int nb, nbj, zero_blk, n_pad, wave, tid;
  int poff;                 // the block produced at step J is J + poff (this pass)
  int pw0, pw1;             // the pass's production window: blocks [pw0, pw1)
  int voff;                 // this lane's byte offset inside a fragment plane
  const _Float16* Kb;       // this lane's B-fragment base inside the ring
  const float* ctile;       // the tile's exact scaled candidate coordinates [NT][D]
};

// B fragments of half h of block J: columns (2h + b)*16 + lane%16, rows
// 8*(lane/16) .. +7.
template <int NT>
__device__ __forceinline__ void load_b(const Ctx& C, int J, int h, BHalf& B) {
  const _Float16* kb = C.Kb + (J % kRing) * kJ;
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    B.hi[b] = *reinterpret_cast<const halfx8*>(kb + (2 * h + b) * 16 * kCSH);
    B.lo[b] = *reinterpret_cast<const halfx8*>(kb + (NT + (2 * h + b) * 16) * kCSH);
  }
}

// One step J for slots [LO, RB). B0 holds the first half of block J's B
// fragments on entry (read during the previous step) and the first half of
// block J + 1's on exit; the second half is read at the start. The MFMAs of
// block J (fragments for J + 1 requested on the way) and the producer's block
// J + 2 (when PROD) are independent and are left to the scheduler to
// interleave: the fp16 MFMAs overlap the VALU work. The step's barrier
// publishes the produced block; block J + 1 was
// published by the previous step's, so its B fragments can be read early.
template <int LO, int RB, int NT, int DX4, bool COMP, bool PROD>
__device__ __forceinline__ void step(const Ctx& C, const PosteriorArgs& a, Producer<NT, DX4, COMP>& P,
                                     _Float16* ring, const Slots<RB>& sl, int J,
                                     BHalf& B0, AFrag (&av)[RB], floatx4 (&acc)[RB][NT / 16]) {
  constexpr int NCB = NT / 16;
  static_assert(NCB == 4, "two halves of two column blocks");
  BHalf B1;
  load_b<NT>(C, J, 1, B1);
  // the distances consume the producer's operands, except alpha and the
  // weights (copied), so the next block's are requested right after them, a
  // whole step before they are needed (requested at the end of the step,
  // they made the next step start by waiting for them)
  using Pr = Producer<NT, DX4, COMP>;
  float r2[Pr::NS][4];
  floatx4 al, wt;
  if constexpr (PROD) {
    produce_dist(P, a, J + C.poff, C.ctile, r2);
    al = P.al;
    wt = P.wt;
  }
  if constexpr (PROD) {
    prod_load(P, C.n_pad, J + 1 + C.poff, C.tid & 63);
  } else {
    // only the step before the first producing one needs them
    const int jn = J + 1 + C.poff;
    if (jn >= C.pw0 && jn < C.pw1) prod_load(P, C.n_pad, jn, C.tid & 63);
  }
  if constexpr (PROD) produce_kv(P, a, J + C.poff, r2, al, wt, ring);
  // slot pairs in turn, each pair's fragments for J + 1 requested as soon as
  // its MFMAs are issued (about half a step before the next step needs them);
  // the next block's first B half is read once the last pair is done with it
#pragma unroll
  for (int r0 = LO; r0 < RB; r0 += 2) {
    mfma_pair_half<RB, NCB, 0>(r0, av, B0, acc);
    if (r0 + 2 >= RB) load_b<NT>(C, J + 1, 0, B0);
    mfma_pair_half<RB, NCB, 1>(r0, av, B1, acc);
#pragma unroll
    for (int r = r0; r < r0 + 2 && r < RB; ++r)
      av[r] = load_a(C.lp_rs, C.voff, frag_block(sl.first[r], sl.last[r], J + 1, C.zero_blk));
  }
  if constexpr (LO >= RB) load_b<NT>(C, J + 1, 0, B0);
  if constexpr (PROD) {
    // interleave: the scheduler otherwise runs the producer's VALU work and
    // the MFMAs as two separate stretches, and the two waves of a SIMD
    // (kept in step by the barriers) then contend for the same unit
    constexpr int nM = 3 * NCB * (RB - LO) + Pr::NS * Pr::NF;
    constexpr int nV = 4 * (COMP ? 40 : 22);
    if constexpr (nM > 0) {
#pragma unroll
      for (int i = 0; i < nM; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, (nV + nM - 1) / nM, 0);  // VALU
      }
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  lds_barrier();
}

// Steps [j0, j1) for slots [LO, RB); the producer runs at the steps whose
// block J + poff lies in the pass's production window [pw0, pw1).
template <int LO, int RB, int NT, int DX4, bool COMP>
__device__ __forceinline__ void span(const Ctx& C, const PosteriorArgs& a, Producer<NT, DX4, COMP>& P,
                                     _Float16* ring, const Slots<RB>& sl, int j0,
                                     int j1, int pw0, int pw1, BHalf& B0, AFrag (&av)[RB],
                                     floatx4 (&acc)[RB][NT / 16]) {
  const int p0 = min(max(pw0 - C.poff, j0), j1), p1 = min(max(pw1 - C.poff, p0), j1);
  int J = j0;
  for (; J < p0; ++J) step<LO, RB, NT, DX4, COMP, false>(C, a, P, ring, sl, J, B0, av, acc);
  for (; J < p1; ++J) step<LO, RB, NT, DX4, COMP, true>(C, a, P, ring, sl, J, B0, av, acc);
  for (; J < j1; ++J) step<LO, RB, NT, DX4, COMP, false>(C, a, P, ring, sl, J, B0, av, acc);
}

// Rounds R.. of the triangular part of a pass: round R covers the row blocks
// base + 8R .. base + 8R + 7, i.e. J in [base/2 + 4R, base/2 + 4R + 4); slot R
// is live while J <= its row block / 2, slots above R throughout.
template <int R, int RB, int NT, int DX4, bool COMP>
__device__ __forceinline__ void rounds(const Ctx& C, const PosteriorArgs& a, Producer<NT, DX4, COMP>& P,
                                       _Float16* ring, const Slots<RB>& sl,
                                       int base, int pw0, int pw1, BHalf& B0, AFrag (&av)[RB],
                                       floatx4 (&acc)[RB][NT / 16]) {
  if constexpr (R < RB) {
    const int j0 = base / 2 + 4 * R;
    if (j0 >= C.nbj) return;
    const int jend = min(j0 + 4, C.nbj);
    const int jlive = min(slot_block(base, R, C.wave) / 2 + 1, jend);
    span<R, RB, NT, DX4, COMP>(C, a, P, ring, sl, j0, jlive, pw0, pw1, B0, av, acc);
    span<R + 1, RB, NT, DX4, COMP>(C, a, P, ring, sl, jlive, jend, pw0, pw1, B0, av, acc);
    rounds<R + 1, RB, NT, DX4, COMP>(C, a, P, ring, sl, base, pw0, pw1, B0, av, acc);
  }
}

template <int NT, int DX4, int Q, int RB, bool COMP>
__global__ __launch_bounds__(kThreads) void k_posterior(PosteriorArgs a) {
  extern __shared__ float smem[];
  constexpr int NCB = NT / 16;          // 16-column blocks per tile
  constexpr int NX = (Q > 1) ? Q : 1;   // per-point partial slots (diag + xors)
  using Prod = Producer<NT, DX4, COMP>;
  static_assert(NT == 64, "eight 16x16 tiles per 32-row block");
  constexpr int D = Prod::D;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // wave index as a scalar: the loop control below stays uniform
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n_pad = a.nb * kBlk;
  _Float16* ring = reinterpret_cast<_Float16*>(smem);       // 2 planes x NT x kCSH halves
  float* red = smem;                                        // kWaves * NT * NX, after the loop
  float* ctile = smem + NT * kCSH;                          // NT * D exact scaled candidates
  float* mush = ctile + NT * D;                             // 2 * NT (mu per row half)
  float* kpp = mush + 2 * NT;                               // NT * 4 (prior cross-cov)
  float* wsh = kpp + NT * 4;                                // NT: w(candidate), composite
  float* kish = wsh + NT;                                   // NT: 2^(E-14) of each column's split scale
  const int64_t p0 = (int64_t)blockIdx.x * NT;

  Prod P;
  float wstar = 0.f;        // composite: w(candidate)
  P.half = wave >> 2;
  P.col = 16 * (wave & 3) + (lane & 15);
  P.rq = 16 * P.half + 4 * (lane >> 4);
  const int64_t pcol = p0 + P.col;
  const bool valid = pcol < a.npts;
  float cc[D];              // this lane's candidate, scaled (slot layout)
#pragma unroll
  for (int t = 0; t < D; ++t) cc[t] = 0.f;
  P.wsd = 0.f;
  if (valid) {
    const float* cp = a.cand + pcol * a.d;
#pragma unroll
    for (int t = 0; t < D; ++t) {
      const int c = slot_dim(t, a.d, a.dr, a.dr4);
      if (c >= 0) cc[t] = cp[c] * a.invls[t];
    }
    if constexpr (COMP) {
      float e = 0.f;
      for (int t = a.dr; t < a.d; ++t) e = fmaf(a.pref[t - a.dr], cp[t], e);
      wstar = expf(e);
      P.wsd = a.s_dep * wstar;
    }
  }
  // power of two for this column's kernel values: a plain model's is uniform
  // (its covariances are bounded by s; the host folds it into a.ss), a
  // composite column's follows from the bound sqrt(prior(candidate) * kbound)
  float kinv = a.kinv0;
  if constexpr (COMP) {
    const KvScale ks = kv_split_scale(
        __builtin_amdgcn_sqrtf(fmaf(a.s_dep * wstar, wstar, a.s + a.s_int) * a.kbound));
    P.wsd *= ks.ksc;
    P.ss = a.s * ks.ksc;
    P.sis = a.s_int * ks.ksc;
    kinv = ks.kinv;
  }
  // distance operands of the candidate: centred coordinates, their squared
  // norms per group, and the B fragments, laid out per group and column in
  // the (not yet used) ring as 96 halves: [0, 32) stream 0 (hi, zero past D),
  // [32, 96) stream 1 (hi at p < D, lo at D <= p < 2D, zero beyond)
  {
    float ct[D];
#pragma unroll
    for (int t = 0; t < D; ++t) ct[t] = cc[t] - a.ctr[t];
#pragma unroll
    for (int g = 0; g < Prod::NS; ++g) {
      float n2 = 0.f;
#pragma unroll
      for (int t = 0; t < D; ++t) {
        const bool in = !COMP || ((t < 4 * a.dr4) == (g == 0));
        if (in) n2 = fmaf(ct[t], ct[t], n2);
      }
      P.c2[g] = n2;
    }
    // a candidate with a non-finite coordinate: its unscale factor is NaN, so
    // its mu and variance read NaN (the hot loop's clamps would hide it)
    if (!(P.c2[0] + P.c2[Prod::NS - 1] < __builtin_huge_valf())) kinv = __builtin_nanf("");
    _Float16* hs = ring;
    if (P.half == 0 && (lane >> 4) == 0) {
#pragma unroll
      for (int g = 0; g < Prod::NS; ++g) {
        _Float16* h = hs + (g * NT + P.col) * 96;
        halfx8 v[12];
#pragma unroll
        for (int i = 0; i < 12; ++i) v[i] = halfx8{};
#pragma unroll
        for (int t = 0; t < D; ++t) {
          const bool in = !COMP || ((t < 4 * a.dr4) == (g == 0));
          const _Float16 hi = static_cast<_Float16>(in ? ct[t] : 0.f);
          const _Float16 lo = static_cast<_Float16>(
              in ? (ct[t] - static_cast<float>(static_cast<_Float16>(ct[t]))) * kDistLoScale : 0.f);
          v[t / 8][t % 8] = hi;
          v[(32 + t) / 8][(32 + t) % 8] = hi;
          v[(32 + D + t) / 8][(32 + D + t) % 8] = lo;
        }
#pragma unroll
        for (int i = 0; i < 12; ++i) *reinterpret_cast<halfx8*>(h + 8 * i) = v[i];
      }
#pragma unroll
      for (int t4 = 0; t4 < DX4; ++t4)
        *reinterpret_cast<float4*>(ctile + P.col * D + 4 * t4) =
            float4{cc[4 * t4], cc[4 * t4 + 1], cc[4 * t4 + 2], cc[4 * t4 + 3]};
      if (COMP) wsh[P.col] = wstar;
      kish[P.col] = kinv;
    }
    __syncthreads();
#pragma unroll
    for (int g = 0; g < Prod::NS; ++g)
#pragma unroll
      for (int f = 0; f < Prod::NF; ++f)
        P.cb[g][f] = *reinterpret_cast<const halfx8*>(hs + (g * NT + P.col) * 96 + 32 * f +
                                                      8 * (lane >> 4));
    // the ring is written from here on
    __syncthreads();
  }

  if (Q > 1) {
    // prior covariance of each point with its batch mates (point ^ x), partner
    // x on the lane of the column (first row half) whose row group is x
    const int x = lane >> 4;
    if (P.half == 0 && x >= 1 && x < Q) {
      const int64_t pm = pcol ^ x;
      float r2 = 0.f, r2r = 0.f, wm = 0.f;     // r2r, wm: composite routing part, w(partner)
      if (valid && pm < a.npts) {
        const float* cp = a.cand + pm * a.d;
#pragma unroll
        for (int t = 0; t < D; ++t) {
          if constexpr (COMP) {
            if (t == 4 * a.dr4) {
              r2r = r2;
              r2 = 0.f;
            }
          }
          const int c = slot_dim(t, a.d, a.dr, a.dr4);
          if (c >= 0) {
            const float dd = cc[t] - cp[c] * a.invls[t];
            r2 = fmaf(dd, dd, r2);
          }
        }
        if constexpr (COMP) {
          float e = 0.f;
          for (int t = a.dr; t < a.d; ++t) e = fmaf(a.pref[t - a.dr], cp[t], e);
          wm = expf(e);
        }
      }
      if constexpr (COMP) {
        // s_route M52(r_route) + s_dep w w' M32(r_dep) + s_int M52 M32
        const float k5 = matern52_f(r2r, 1.0f);
        const float k3 = matern32_f(r2);
        kpp[P.col * 4 + x] = fmaf(a.s_dep * wstar * wm, k3, k5 * fmaf(a.s_int, k3, a.s));
      } else {
        kpp[P.col * 4 + x] = matern52_f(r2, a.s);
      }
    }
  }

  Ctx C;
  C.nb = a.nb;
  C.nbj = (a.nb + 1) / 2;
  C.zero_blk = frag_row_start(a.nb);
  C.lp_rs = make_rsrc(a.Lp, (C.zero_blk + 1) * 2048 + 4 * (a.nb + 1));
  P.xf_rs = make_rsrc(a.xf, a.nb * Prod::NF * 1024);
  P.x2_rs = make_rsrc(a.x2, 2 * n_pad * 4);
  P.al_rs = make_rsrc(a.alpha, n_pad * 4);
  P.xs_rs = make_rsrc(a.Xs, n_pad * a.dx * 4);
  if constexpr (COMP) P.wt_rs = make_rsrc(a.wts, n_pad * 4);
  C.n_pad = n_pad;
  C.wave = wave;
  C.tid = tid;
  C.ctile = ctile;
  C.voff = lane * 16;
  // B fragments: column (b*16 + lane%16), rows 8*(lane/16) .. +7 of a block
  C.Kb = ring + (lane & 15) * kCSH + 8 * (lane >> 4);

  float ss[NCB];
  float gx[NCB][NX];
#pragma unroll
  for (int b = 0; b < NCB; ++b) {
    ss[b] = 0.f;
#pragma unroll
    for (int x = 0; x < NX; ++x) gx[b][x] = 0.f;
  }

  // blocks 0 .. have-1 of K*^T are in the ring (have = 0: start over)
  int have = 0;
  for (int base = 0; base < a.nb; base += 8 * RB) {
    const int jpass = min(C.nbj, base / 2 + 4 * RB);   // J range of this pass
    floatx4 acc[RB][NCB];
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
      for (int b = 0; b < NCB; ++b) acc[r][b] = floatx4{0.f, 0.f, 0.f, 0.f};
    Slots<RB> sl;
    AFrag av[RB];
    // the slots' row-block scales, stored after the packed fragments (and the
    // zero block): entry I < nb, and a zero at nb for slots past the matrix.
    // Loaded into vector registers: held in scalar ones across the pass they
    // would spill.
    float scv[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int I = slot_block(base, r, wave);
      sl.first[r] = I < a.nb ? frag_row_start(I) : C.zero_blk;
      sl.last[r] = I < a.nb ? I / 2 : -1;
      scv[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
          C.lp_rs, 4 * min(I, a.nb) + 0 * lane, (C.zero_blk + 1) * 2048, 0));
      av[r] = load_a(C.lp_rs, C.voff, frag_block(sl.first[r], sl.last[r], 0, C.zero_blk));
    }
    // Production schedule. Starting over, blocks 0 and 1 are made here and
    // block J + 2 at step J (poff = 2). A pass that finds blocks 0..have-1
    // in the ring makes block have - 1 + J at step J >= 1 (poff = have - 1),
    // into the slot of block J - 1, which no wave reads after step J - 1:
    // the new blocks are made during the pass's first steps, where every
    // slot is live and the matrix cores have the most work to hide them
    // behind. The operands of a block are loaded a step before it is made.
    const int have0 = have;
    if (have == 0) {
      // start over: blocks 0 and 1, and mu from scratch
      P.mu = 0.f;
      prod_load(P, n_pad, 0, lane);
      produce(P, a, 0, ctile, ring);
      prod_load(P, n_pad, 1, lane);
      produce(P, a, 1, ctile, ring);
      have = 2;
      lds_barrier();
    }
    C.poff = have0 ? have0 - 1 : 2;
    prod_load(P, n_pad, C.poff, lane);   // block poff: made at step 0 when new
    const int pw0 = have, pw1 = jpass;   // blocks this pass produces
    C.pw0 = pw0;
    C.pw1 = pw1;
    BHalf B0;
    load_b<NT>(C, 0, 0, B0);
    // blocks left of this pass's triangle: every slot is live
    span<0, RB, NT, DX4, COMP>(C, a, P, ring, sl, 0, base / 2, pw0, pw1, B0, av, acc);
    rounds<0, RB, NT, DX4, COMP>(C, a, P, ring, sl, base, pw0, pw1, B0, av, acc);
    have = (jpass <= kRing) ? max(have, jpass) : 0;

    // undo the row-block scale of L^{-1} (the column scale of K*^T is undone
    // per point in the epilogue); slots past the matrix hold zeros
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const float sc = scv[r];
#pragma unroll
      for (int b = 0; b < NCB; ++b)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float v = acc[r][b][e] * sc;
          ss[b] = fmaf(v, v, ss[b]);
          if (Q > 1) {
#pragma unroll
            for (int x = 1; x < NX; ++x) gx[b][x] = fmaf(v, quad_xor(v, x), gx[b][x]);
          }
        }
    }
  }

  // mu: the last pass produced every block; reduce over the lanes of a column
  {
    float v = P.mu;
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    if (lane < 16) mush[P.half * NT + P.col] = v;
  }
  // |v|^2 (and cross terms): over the four 16-lane row groups, then over
  // waves in LDS (red overlays the ring: wait until every wave is done)
  __syncthreads();
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
    // undo the columns' kernel-value scales: |v|^2 carries ki^2, a cross
    // product with batch mate tid ^ x carries ki times the mate's
    const float ki = kish[tid];
#pragma unroll
    for (int x = 1; x < NX; ++x) tot[x] = (tot[x] * ki) * kish[tid ^ x];
    const float mu = (mush[tid] + mush[NT + tid]) * ki;
    float var;
    if constexpr (COMP) {
      const float w = wsh[tid];
      const float prior = fmaf(a.s_dep * w, w, a.s + a.s_int);     // s_route + s_dep w*^2 + s_int
      var = prior - (tot[0] * ki) * ki;
    } else {
      // in the column's scaled units (s 2^(14-E) - |v|^2 2^(14-E)), then
      // unscaled: the same rounding as s - |v|^2
      var = (a.ss - tot[0] * ki) * ki;
    }
    if (valid) {
      a.mu[p * a.mu_ps] = mu;
      // clamp at zero; a NaN variance stays NaN
      a.sd[p * a.sd_ps] = __builtin_amdgcn_sqrtf(var < 0.f ? 0.f : var);
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
        // pivot scale: the prior scale (composite: the sum of the three)
        const float tol = 1e-10f * (COMP ? a.s + a.s_dep + a.s_int : a.s);
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
          } else if (pv != pv) {
            L[j][j] = pv;     // a NaN pivot stays NaN
          }
        }
        constexpr int T = Q * (Q + 1) / 2;
        float* dst = a.chol + bat * T;
#pragma unroll
        for (int i = 0; i < Q; ++i)
#pragma unroll
          for (int j = 0; j <= i; ++j) dst[i * (i + 1) / 2 + j] = L[i][j];
      }
    }
  }
}

constexpr size_t lds_floats(int NT, int DX4, int q) {
  // ring: 2 planes x NT columns x kCSH halves (the reduction and, before the
  // loop, the candidates' distance fragments overlay it); the exact scaled
  // candidates; mu per row half, the prior cross-covariances, the
  // candidates' preference weights and their kernel-value scales
  return (size_t)NT * kCSH + (size_t)NT * 4 * DX4 + 2 * NT + (size_t)NT * 4 + 2 * NT;
}
static_assert((size_t)kWaves * 64 * 4 <= (size_t)64 * kCSH, "reduction fits the ring");
static_assert(2 * 64 * 96 <= 2 * 64 * kCSH, "distance fragments fit the ring");

template <int NT, int DX4, int Q, int RB, bool COMP>
hipError_t launch_t(const PosteriorArgs& a, hipStream_t st) {
  const size_t lds = sizeof(float) * lds_floats(NT, DX4, Q);
  // more than 64 KiB of dynamic LDS: opt in (cheap; set on every launch so
  // that it holds on whichever device is current)
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_posterior<NT, DX4, Q, RB, COMP>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     static_cast<int>(lds));
  if (e != hipSuccess) return e;
  const unsigned grid = static_cast<unsigned>((a.npts + NT - 1) / NT);
  hipLaunchKernelGGL((k_posterior<NT, DX4, Q, RB, COMP>), dim3(grid), dim3(kThreads), lds, st, a);
  return hipGetLastError();
}

// Launch for coordinate width 4*DX4 and kernel family COMP: q in {1, 2, 4};
// 2 row-block slots per wave up to 256 rows, else BO_POST_RB (further rows
// in passes).
template <int DX4, bool COMP>
hipError_t launch_for_dx(const PosteriorArgs& a, hipStream_t st) {
  const bool small = a.nb <= 16;
  switch (a.q) {
    case 1: return small ? launch_t<BO_POST_NT, DX4, 1, 2, COMP>(a, st)
                         : launch_t<BO_POST_NT, DX4, 1, BO_POST_RB, COMP>(a, st);
    case 2: return small ? launch_t<BO_POST_NT, DX4, 2, 2, COMP>(a, st)
                         : launch_t<BO_POST_NT, DX4, 2, BO_POST_RB, COMP>(a, st);
    case 4: return small ? launch_t<BO_POST_NT, DX4, 4, 2, COMP>(a, st)
                         : launch_t<BO_POST_NT, DX4, 4, BO_POST_RB, COMP>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

// One per coordinate width and kernel family (posterior_dx<N>.hip: Matern-5/2,
// posterior_dx<N>c.hip: composite kernel; a composite model needs at least two
// coordinate groups, so width 4 has no composite instantiation).
hipError_t launch_posterior_dx1(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_dx2(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_dx3(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_dx4(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_dx5(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_dx6(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_dx7(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_dx8(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_comp_dx2(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_comp_dx3(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_comp_dx4(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_comp_dx5(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_comp_dx6(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_comp_dx7(const PosteriorArgs& a, hipStream_t st);
hipError_t launch_posterior_comp_dx8(const PosteriorArgs& a, hipStream_t st);

}  // namespace bo
