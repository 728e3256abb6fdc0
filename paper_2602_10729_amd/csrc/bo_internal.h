// Internal declarations shared by the host API and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/bo.h"

namespace bo {

// Tile geometry of the scoring path.
constexpr int kBlk = 16;        // MFMA 16x16x4 fp32 block edge
constexpr int kFitBlk = 64;     // Cholesky / inverse block edge (fp64)

// Scratch of the no-allocation scoring entry point (noalloc.hip): 32 MiB
// per device, the boxes first (room for BO_MAX_BOXES boxes of three
// objectives), then the posterior workspace.
constexpr size_t kNoallocScratchFloats = (size_t)32 << 18;          // 32 MiB
constexpr size_t kNoallocBoxFloats = (size_t)BO_MAX_BOXES * 2 * 3;
// Device address of this device's scratch (the device must be current);
// looked up once per device with hipGetSymbolAddress.
bo_status noalloc_scratch(int dev, float** out);

// Thread-local error detail; returns the status for chaining.
bo_status fail(bo_status st, const std::string& msg);
bo_status hip_fail(hipError_t e, const char* what);

// Host geometry (host_geom.cpp) -------------------------------------------
// Non-dominated rows of Y (maximise, duplicates keep the lowest index),
// optionally only rows strictly above ref, sorted by objective 0 then index.
// (instantiated for float and double)
template <typename T>
void host_front(const T* Y, int64_t n, int m, const T* ref, std::vector<int32_t>& out);
// Disjoint boxes of the region the front does not dominate; lo/hi row-major
// [count][m]; hi may be +inf.
template <typename T>
void host_boxes(const T* F, int P, int m, const T* ref, std::vector<T>& lo, std::vector<T>& hi);

// Device layout of a fitted model ----------------------------------------
struct Model {
  int device = 0;
  int64_t n = 0;
  int d = 0, m = 0;
  int n_pad = 0;                 // n rounded up to kBlk
  int nb = 0;                    // n_pad / kBlk
  int dx = 0;                    // padded coordinate stride (multiple of 4)
  // composite kernel (dr > 0): routing coordinates 0..dr-1 sit in slots
  // 0..4*dr4-1 of the scaled layout, deployment coordinates from slot 4*dr4
  int dr = 0, dr4 = 0;
  std::vector<float> ls, os, noise;   // os: the (routing) output scale
  std::vector<float> s_dep, s_int;    // composite: deployment / interaction scales
  std::vector<float> prefh;           // composite: host copy of pref [m][d - dr]
  std::vector<float> Yh;         // host copy of Y [n][m]
  std::vector<int32_t> nd;       // non-dominated rows (no reference filter)

  // one device allocation holds every buffer the fit writes (Xs .. ils64,
  // wts, pref below are views into it)
  unsigned char* arena = nullptr;
  size_t arena_bytes = 0;
  // device work that reads the model's buffers may be pending (set while the
  // fit runs and by every call that uses the model; cleared when the fit has
  // synchronised): releasing then waits for the device first
  bool pending = false;
  float* Xs = nullptr;           // [m][n_pad][dx] X / lengthscale (fp32)
  float* invls = nullptr;        // [m][dx] 1 / lengthscale (fp32, 0-padded)
  float* alpha = nullptr;        // [m][n_pad]
  float* wts = nullptr;          // composite: [m][n_pad] preference weights of X (0 past n)
  float* pref = nullptr;         // composite: [m][d - dr] preference slopes
  float* Lp = nullptr;           // [m][lp_per_obj]: packed fp16 hi/lo L^{-1} blocks, the zero
                                 // block, then the nb row-block scales (packed_factor_floats)
  size_t lp_per_obj = 0;         // floats per objective in Lp
  std::vector<float> kbound;     // [m] largest diagonal of K (bounds every training prior variance)
  std::vector<double> cond_est;  // [m] max K_ii * max |L^{-1}|^2 (a lower bound on cond(K))
  // fp64 scoring (bo_fit_f64 / bo_fit_composite_f64): L^{-1} as fp64 MFMA
  // fragments, alpha and the inverse lengthscales in fp64; the raw X is Xd
  bool f64 = false;
  double* Lp64 = nullptr;        // [m][posterior_f64_blocks(nb)][512]
  double* alpha64 = nullptr;     // [m][n_fit]
  double* ils64 = nullptr;       // [m][d]
  int n_fit = 0;
  uint16_t* xf = nullptr;        // [m][nb][dist_frags(dx)][512] distance fragments of X
  float* x2 = nullptr;           // [m][2][n_pad] squared norms of the centred rows
  float* ctr = nullptr;          // [m][dx] centre of the scaled coordinates

  // scoring workspace (grown on demand)
  float* ws = nullptr;
  size_t ws_floats = 0;
  // noisy acquisition (bo_nehvi_prepare): per-sample fronts and the factors
  // of the in-sample conditional
  struct Noisy {
    int S = 0, Sp = 0, n32 = 0, total = 0;
    float* Lp0 = nullptr;        // [m][lp_per_obj] packed inverse factor of K_XX (no noise)
    uint16_t* Gp = nullptr;      // [m][n32][Sp/16][1024] fp16 hi/lo fragments of G^T
    int m = 0, q = 1;            // objectives; batch size of the last scoring call
    float ginv[3] = {1.f, 1.f, 1.f};  // 1 / scale applied to G before the split
    float* boxes = nullptr;      // [total][2m] per-sample boxes (lo, width), sample s at off[s]
    int* off = nullptr;          // [S + 1]
    int32_t* front = nullptr;    // [S][n] per-sample front indices, sorted by objective 0
    std::vector<int> counts;     // [S] boxes per sample
    std::vector<int> fsize;      // [S] front size per sample
    bool cons = false;
    float low[3] = {0.f, 0.f, 0.f};
    float* ws = nullptr;         // scoring workspace
    size_t ws_floats = 0;
  } nz;
  float* Xd = nullptr;           // [n][d] copy of the training inputs

  // box cache (rebuilt when the reference point changes)
  float* d_boxes = nullptr;      // [nbox][2m]: lo then width
  int box_cap = 0;
  int nbox = -1;
  std::vector<float> box_ref;
  // the model's last asynchronous call: a call on another stream waits for it
  hipStream_t last_stream = nullptr;
  hipEvent_t last_evt = nullptr;
};

// Kernel launchers (fit.hip / posterior.hip / ehvi.hip / argmax.hip) -------
// All return hipSuccess or the launch error.

// Kernel hyperparameters on the device (fp64). Plain Matern-5/2: dr = 0 and
// only ils, os, noise are read; composite: os is the routing scale and
// s_dep, s_int, pref [m][d - dr] are read too.
struct GramParams {
  int dr = 0;
  const double* ils = nullptr;     // [m][d] 1 / lengthscale
  const double* os = nullptr;      // [m]
  const double* noise = nullptr;   // [m]
  const double* s_dep = nullptr;   // [m]
  const double* s_int = nullptr;   // [m]
  const double* pref = nullptr;    // [m][d - dr]
};
// Gram matrices K_k + eta_k I in fp64 for all objectives, padded to
// n_fit x n_fit with an identity tail; only the lower block triangle (64x64
// blocks) is written. A: [m][n_fit][n_fit].
// kdiag (optional, [m], zeroed by the caller): the largest diagonal entry of
// each objective's K, as the bit pattern of a non-negative double.
// [col0, col1) (multiples of 16; col1 < 0: n_fit) limits the launch to those
// columns, so the matrix can be written in parts.
hipError_t launch_gram(const float* X, int64_t n, int d, int m, int n_fit,
                       const GramParams& g, double* A, hipStream_t st,
                       unsigned long long* kdiag = nullptr, int col0 = 0, int col1 = -1);
// Composite: wts[k][i] = fp32(exp(sum_j pref[k][j] X[i][dr + j])), 0 for
// n <= i < n_pad.
hipError_t launch_weights(const float* X, int64_t n, int d, int m, int n_pad,
                          const GramParams& g, float* wts, hipStream_t st);
// Blocked right-looking Cholesky of m matrices [m][nf][nf] (lower, in place);
// also leaves W = L^{-1} in W's lower 64-blocks ([m][nf][nf]; W needs no
// initial contents, its blocks above the diagonal are left as they were).
// *flag is set non-zero on a non-positive or non-finite pivot.
// before_update (optional): an event the stream waits for after the first
// diagonal block and its panel and before the first trailing update (which
// reads the columns past the first 64), so that those columns may still be
// in production on another stream when this is called.
hipError_t launch_cholesky(double* A, double* W, int nf, int m, int* flag,
                           hipStream_t st, hipEvent_t before_update = nullptr);
// alpha_k = W_k^T (W_k y_k), y from Y [n][m] (fp32), written fp32 [m][n_pad]
// (and, when alpha64 is not NULL, fp64 [m][nf]). tmp [m][nf] keeps W_k y_k.
hipError_t launch_alpha(const double* W, const float* Y, int64_t n, int m,
                        int nf, int n_pad, double* tmp, float* alpha,
                        hipStream_t st, double* alpha64 = nullptr);
// Log marginal likelihood parts and gradient (fp64) from the factored fit
// scratch: A holds L (lower), W = L^{-1}, tmp = W y, alpha64 = K^{-1} y.
// Overwrites A's lower 64-blocks with K^{-1} = W^T W. partials:
// [m][tiles16][d + 2] scratch with tiles16 = mll_tiles(nf); out [m][1 + d + 2]
// = (value, gradient).
int64_t mll_tiles(int nf);
hipError_t launch_mll(const float* X, int64_t n, int d, int m, int nf, const GramParams& g,
                      double* A, const double* W, const double* tmp, const double* alpha64,
                      double* partials, double* out, hipStream_t st);
// The lengthscale-scaled X in the slot layout from the fp64 inverse
// lengthscales ils [m][d], with the fp32 per-slot values invls [m][dx], the
// copy Xd [n][d] of X, (composite, pref non-NULL) the fp32 preference slopes
// pref [m][d - dr] from their fp64 copies pref_d, and (ils64 non-NULL) a copy
// of ils.
hipError_t launch_scale_x(const float* X, int64_t n, int d, int m, int nb, int dx, int dr,
                          int dr4, const double* ils, float* invls, const double* pref_d,
                          float* pref, float* Xd, double* ils64, float* Xs, hipStream_t st);

// Squared distances in the posterior kernel come from the expansion
// |c|^2 + |x|^2 - 2 c.x of centred scaled coordinates, with c.x on the fp16
// matrix cores: each value splits into hi = fp16(v) and lo = fp16(2^11 (v -
// hi)); one accumulator takes sum x_hi c_hi over the D = dx slots (stream 0),
// another sum x_lo c_hi + x_hi c_lo over 2D positions (stream 1), and c.x =
// acc0 + 2^-11 acc1. Fragments of 32 k-positions per 16-row group: stream 0
// first, then stream 1.
__host__ __device__ constexpr int dist_frags0(int dx) { return (dx + 31) / 32; }
__host__ __device__ constexpr int dist_frags(int dx) { return (dx + 31) / 32 + (2 * dx + 31) / 32; }
constexpr float kDistLoScale = 2048.0f;

// Centre the scaled coordinates (ctr = mean over the n rows), then write the
// A fragments of the centred rows (xf, zero for rows past n) and their
// squared norms per coordinate group (x2 [2][n_pad]: routing slots t < 4*dr4,
// then the rest; a plain model has everything in the second group).
hipError_t launch_pack_x(const float* Xs, int64_t n, int m, int nb, int dx, int dr4,
                         float* ctr, uint16_t* xf, float* x2, hipStream_t st);

// Noisy acquisition, fp64 preparation (fit.hip).
// A holds K^{-1} in its lower 64-blocks on return (from W = L^{-1}).
hipError_t launch_kinv(double* A, const double* W, int nf, int m, hipStream_t st);
// A (lower 64-blocks, K^{-1} on entry) <- eta (I - eta K^{-1}), identity tail.
hipError_t launch_sigma_xx(double* A, int64_t n, int nf, int m, const double* noise,
                           hipStream_t st);
// Zk[k][i][s] = ZX[s][i][k] (fp64 [m][nf][Sp], zero-padded).
hipError_t launch_gather_z(const float* ZX, int64_t n, int m, int S, int nf, int Sp,
                           double* Zk, hipStream_t st);
// C[k] = op(T[k]) Bm[k]: T lower [nf][nf], Bm and C [nf][ldb], op = T or T^T.
hipError_t launch_trmm(bool trans, const double* T, const double* Bm, double* C, int nf,
                       int ldb, int m, hipStream_t st);
// Pack W into the posterior's A-fragment format (fp16 hi/lo planes of 16x32
// lower blocks, zeros beyond n, then one all-zero block; 2 KiB per block,
// posterior_frag_blocks(nb) blocks per objective), each 16-row block I scaled
// by a power of two that brings its largest entry into [2^13, 2^14), followed
// by the nb inverse scales (packed_factor_floats(nb) floats per objective;
// wmax [m] = largest |W| per objective as a non-negative double's bit
// pattern, zeroed by the caller; *flag set on a non-finite entry).
// bmax (optional, [m][nb], zeroed by the caller): the row-block maxima are
// gathered there by column chunks (more workgroups, for the fit's critical
// path) and the pack derives the scales from them.
hipError_t launch_pack_factor(const double* W, int64_t n, int m, int nf, int nb, float* Lp,
                              unsigned long long* wmax, int* flag, hipStream_t st,
                              unsigned long long* bmax = nullptr);

// Noisy acquisition kernels (nehvi.hip).
struct NehviFrontArgs {
  const float* Y;          // [n][2] observations (fp32)
  const double* alpha64;   // [2][nf] K^{-1} y
  const double* noise;     // [2] noise variances
  const double* T1;        // [2][nf][Sp] L_XX Z_X
  int64_t n;
  int nf, Sp, S;
  float ref0, ref1;
  bool cons;
  float low0, low1;
  float* boxes;            // [S][n + 1][4]
  int* counts;             // [S] boxes per sample
  int32_t* front;          // [S][n]
};
hipError_t launch_sample_fronts(const NehviFrontArgs& a, hipStream_t st);
// Per-sample fronts and boxes of three objectives (k_sample_front3).
struct NehviFront3Args {
  const double* F;         // [S][n][3] in-sample draws
  int64_t n;
  int S;
  float ref[3];
  bool cons;
  float low[3];
  float* boxes;            // [S][3n + 1][6]
  int* counts;             // [2S]: boxes, then front size, per sample
  int32_t* front;          // [S][n]
  int* bad;                // set to 1 on a non-finite draw
};
hipError_t launch_sample_fronts3(const NehviFront3Args& a, hipStream_t st);
size_t nehvi_front3_lds_bytes(int64_t n);
hipError_t launch_compact_boxes3(const float* tmp, int64_t stride, const int* off, int S,
                                 float* out, hipStream_t st);
// F[s][i][k] = y_ik - eta_k alpha_k,i + T1[k][i][s] (fp64, the in-sample draws)
hipError_t launch_insample_values(const float* Y, const double* alpha64, const double* noise,
                                  const double* T1, int64_t n, int m, int nf, int Sp, int S,
                                  double* F, hipStream_t st);
size_t nehvi_front_lds_bytes(int64_t n);
// part [m][kAbsmaxParts]: partial maxima of |G[k]| (count entries per objective)
constexpr int kAbsmaxParts = 128;
hipError_t launch_absmax(const double* G, int64_t count, int m, double* part, hipStream_t st);
hipError_t launch_pack_g(const double* G, int nf, int Sp, int n32, int m, const float* scale,
                         uint16_t* Gp, hipStream_t st);
hipError_t launch_compact_boxes(const float* tmp, int64_t stride, const int* off, int S,
                                float* out, hipStream_t st);
struct NehviMeansArgs {
  const float* cand;       // [npts][d]
  int64_t npts;
  int d, dx, n32, n_pad, S;
  const float* Xs;         // [m][n_pad][dx] scaled training inputs
  const float* invls;      // [m][dx]
  const uint16_t* xf;      // [m][xf_stride] centred-X distance fragments (fp16 bits)
  int64_t xf_stride;
  const float* x2;         // [m][2][n_pad] squared norms of the centred rows per group
  const float* ctr;        // [m][dx] centre of the scaled coordinates
  const uint16_t* Gp;      // packed G^T fragments (fp16 bits)
  float s[3];              // output scales (composite: of the routing term)
  float kbound[3];         // composite: bound on every training point's prior variance
  float ginv[3];           // 1 / scale of G
  float* out;              // [m][S][ldo]
  int64_t ldo;
  // composite kernel (dr > 0): slot layout, scales and preference weights
  int dr = 0, dr4 = 0;
  float s_dep[3] = {0.f, 0.f, 0.f}, s_int[3] = {0.f, 0.f, 0.f};
  const float* wts = nullptr;    // [m][n_pad] weights of the training points
  const float* pref = nullptr;   // [m][d - dr] preference slopes
};
hipError_t launch_nehvi_means(const NehviMeansArgs& a, int m, hipStream_t st);
struct NehviEhviArgs {
  const float* mu;         // [m][nbat * q] posterior mean (planar)
  const float* sd;         // q = 1: [m][nbat] noise-free conditional std (tau)
  const float* chol;       // q > 1: [m][nbat][q(q+1)/2] factor of the conditional batch covariance
  const float* D;          // [m][S][ldd] K* G (point index b * q + member)
  int64_t ldd;
  const float* Z;          // [S][q][m] candidate base samples
  const float* boxes;      // [total][2m] (lo, width)
  const int* off;          // [S + 1]
  int total;
  int64_t nbat;
  int S, q, m;
  bool cons;
  float low[3];
  float* ehvi;             // [nbat]
};
hipError_t launch_nehvi_ehvi(const NehviEhviArgs& a, hipStream_t st);
size_t nehvi_ehvi_lds_bytes(int S, int q, int m, int total, bool boxes_in_lds);
int nehvi_padded_samples(int S);

// Coordinate held by slot t of the scaled layout, or -1 for padding: the
// identity for plain models (dr = dr4 = 0); for composite ones the routing
// coordinates fill slots 0..dr-1 (zero up to 4*dr4) and the deployment
// coordinates start at slot 4*dr4.
__host__ __device__ inline int slot_dim(int t, int d, int dr, int dr4) {
  if (t < 4 * dr4) return t < dr ? t : -1;
  const int c = dr + t - 4 * dr4;
  return c < d ? c : -1;
}
// Convert a fp64 [n][n] lower factor (leading dimension nf) to fp32 [n][n].
hipError_t launch_lower_to_f32(const double* A, int64_t n, int nf, float* L,
                               hipStream_t st);
// Copy a fp32 [n][n] matrix into a fp64 padded [nf][nf] with identity tail.
hipError_t launch_f32_to_padded(const float* A, int64_t n, int nf, double* P,
                                hipStream_t st);

// Posterior of one objective for npts points (q consecutive points form a
// batch). Writes mu/var (q = 1) or mu + packed chol factor (q > 1) into the
// workspace arrays described in posterior.hip.
struct PosteriorArgs {
  const float* cand;   // [npts][d]
  int64_t npts;
  int d, dx, q;
  const float* Xs;     // [n_pad][dx]
  const float* invls;  // [dx]
  const float* alpha;  // [n_pad]
  const float* Lp;     // packed fragments of this objective, then its row-block scales
  float kbound;        // composite: bound on every training point's prior variance
  // plain Matern-5/2: the output scale times the kernel values' power-of-two
  // split scale 2^(14 - E) (s = f 2^E, f in [0.5, 1)), and 2^(E - 14)
  float ss, kinv0;
  const uint16_t* xf;  // [nb][dist_frags(dx)][512] centred-X distance fragments
  const float* x2;     // [2][n_pad] squared norms of the centred rows per coordinate group
  const float* ctr;    // [dx] centre subtracted from the scaled coordinates
  int n, nb;
  float s;             // output scale (composite: of the routing term)
  int m, k;            // objective count / index (output strides)
  int dr, dr4;         // composite kernel (dr > 0): routing coordinates / slot chunks
  float s_dep, s_int;  // composite: deployment and interaction scales
  const float* wts;    // composite: [n_pad] preference weights of the training points
  const float* pref;   // composite: [d - dr] preference slopes
  // fp64 scoring: packed fp64 fragments, alpha and 1 / lengthscale of this
  // objective, and the raw training inputs [n][d]
  const double* Lp64 = nullptr;
  const double* alpha64 = nullptr;
  const double* ils64 = nullptr;
  const float* Xraw = nullptr;
  // outputs of this objective: mu and the marginal std of point p at
  // mu[p * mu_ps] and sd[p * sd_ps] (1 for a planar workspace, m for the
  // caller's [npts][m] arrays; the pointers are already at the objective)
  float* mu;
  float* sd;
  int64_t mu_ps = 1, sd_ps = 1;
  float* chol;         // q > 1: [npts/q][q(q+1)/2] lower factors of this objective, row-major
};
hipError_t launch_posterior(const PosteriorArgs& a, hipStream_t st);
// The fp64 posterior (posterior_f64.hip): same outputs, from Lp64, alpha64,
// ils64 and Xraw.
hipError_t launch_posterior_f64(const PosteriorArgs& a, hipStream_t st);
// Blocks per objective of the fp64 fragments (lower 16x32 blocks).
int64_t posterior_f64_blocks(int nb);
// Pack W = L^{-1} ([m][nf][nf] fp64) as the fp64 kernel's A fragments.
hipError_t launch_pack_f64(const double* W, int64_t n, int m, int nf, int nb, double* Lp64,
                           hipStream_t st);
// Packed L^{-1} blocks per objective (lower 16x32 blocks + the zero block).
int64_t posterior_frag_blocks(int nb);
// Floats per objective of the packed inverse factor: the fragment blocks
// (512 floats each), then the nb row-block scales and a zero (the scale of
// a row block past the matrix), padded to 64 floats.
inline size_t packed_factor_floats(int nb) {
  return (size_t)posterior_frag_blocks(nb) * 512 + (size_t)(nb + 1 + 63) / 64 * 64;
}

// Monte-Carlo EHVI over boxes for nbat batches.
struct EhviArgs {
  // mu and sd of objective k at point p: mu[p * mu_ps + k * mu_ks] (planar
  // workspace: ps = 1, ks = nbat*q; the caller's [nbat*q][m]: ps = m, ks = 1)
  const float* mu;
  const float* sd;     // (q = 1)
  int64_t mu_ps, mu_ks, sd_ps, sd_ks;
  const float* chol;   // [m][nbat][q(q+1)/2] (q > 1)
  const float* Z;      // [S][q][m]
  const float* boxes;  // [nbox][2m] lo then width
  int64_t nbat;
  int q, m, S, nbox;
  bool constrained;    // weight samples by feasibility (y_k >= lower[k] for all k)
  float lower[3];      // feasibility thresholds (-inf: objective unconstrained)
  float* ehvi;         // [nbat]
};
hipError_t launch_ehvi(const EhviArgs& a, hipStream_t st);

hipError_t launch_argmax(const float* v, int64_t M, int64_t* index,
                         float* value, hipStream_t st);

// Achieved-peak probes (peaks.hip); synchronous.
hipError_t measure_peak(int what, int64_t iters, double* rate, hipStream_t st);

}  // namespace bo
