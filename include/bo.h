/*
 * bo.h — C ABI of the batch acquisition scorer (MI355X / gfx950).
 *
 * Scores a large batch of encoded candidate configurations for one iteration
 * of multi-objective Bayesian optimisation, as in the online phase of BOute
 * (Jiang, Fu, Yoneki — "BOute: Cost-Efficient LLM Serving with Heterogeneous
 * LLMs and GPUs via Multi-Objective Bayesian Optimization"):
 *
 *   bo_fit    — condition one GP per objective on the observations
 *               (workflow step (i), "Surrogate model fitting"; ARD
 *               Matern-5/2 kernel with an output scale, implementation
 *               section "MOBO optimization kernels"); bo_fit_composite
 *               with the paper's additive, preference-weighted kernel.
 *   bo_score  — GP posterior of every candidate plus Monte-Carlo expected
 *               hypervolume improvement against the Pareto front
 *               (workflow step (ii) and the "Constrained qNEHVI" paragraph:
 *               expectation of HVI over samples of the joint posterior).
 *   bo_argmax — index of the best candidate ("selecting the next candidate
 *               configuration theta*").
 *   bo_score_constrained — bo_score with the feasibility indicator of the
 *               constrained form.
 *   bo_nehvi_prepare / bo_score_nehvi — the noisy form (qNEHVI): the latent
 *               objectives at the observations are sampled jointly with the
 *               candidates, with a Pareto front per sample.
 *   bo_mll    — exact log marginal likelihood and its gradient, for fitting
 *               the hyperparameters on the host.
 *
 * Conventions shared by every entry point:
 *   - All floating-point arrays are fp32, row-major, contiguous.
 *   - "device" pointers are HIP device memory on the current device; "host"
 *     pointers are ordinary host memory read before the call returns.
 *   - The caller owns every buffer it passes; the library never frees them.
 *     Asynchronous calls read/write caller buffers when the stream reaches
 *     the work, so the caller keeps them alive until then.
 *   - stream is a hipStream_t passed as void*; NULL means the null stream.
 *   - Every function returns a status; nothing throws or aborts across the
 *     ABI. Arguments are validated before any device work is enqueued.
 *     bo_last_error_message() gives a thread-local detail string.
 *   - Objectives are maximised and live in standardised units (the caller
 *     standardises Y; the reference point and EHVI are in the same units).
 *   - Kernel faults of an asynchronous call surface at the next synchronous
 *     call; setting BO_SYNC_DEBUG=1 synchronises and checks after each launch.
 *
 * Thread safety: distinct models may be used from distinct threads. Calls
 * that share a model must be ordered by the caller (same stream, or
 * synchronised), because a model keeps one scoring workspace.
 */
#ifndef BO_H_
#define BO_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct bo_model_s* bo_model;   /* opaque, owned by the library */

typedef enum {
  BO_OK = 0,
  BO_ERR_INVALID_ARGUMENT = 1,      /* bad size, null pointer, bad hyperparameter */
  BO_ERR_NOT_POSITIVE_DEFINITE = 2, /* Cholesky pivot <= 0 or non-finite      */
  BO_ERR_CAPACITY = 3,              /* n, d, S or box count beyond compiled limits */
  BO_ERR_DEVICE = 4,                /* a HIP runtime call failed               */
  BO_ERR_OUT_OF_MEMORY = 5,         /* device or host allocation failed        */
  BO_ERR_NONFINITE_INPUT = 6,       /* NaN/Inf in a host-side input            */
  BO_ERR_ILL_CONDITIONED = 7        /* K too ill-conditioned for fp32-class scoring */
} bo_status;

/* Compiled limits (BO_ERR_CAPACITY beyond them). */
#define BO_MAX_N 2048        /* observations                                 */
#define BO_MAX_D 32          /* encoded dimensions                           */
#define BO_MAX_S 4096        /* Monte-Carlo samples                          */
#define BO_MAX_BOXES 4096    /* boxes of the non-dominated region            */

/*
 * bo_fit — exact GP conditioning, one independent GP per objective.
 *
 * Paper: workflow step (i) and the implementation section (one
 * SingleTaskGP per objective combined as a model list; ARD Matern-5/2 in a
 * scale kernel). Hyperparameters are given, not learned.
 *
 * For each objective k (s = outputscale[k], eta = noise[k],
 * l = lengthscale[k*d .. k*d+d-1]):
 *   k(u,v) = s (1 + sqrt5 r + 5/3 r^2) exp(-sqrt5 r),
 *            r = sqrt(sum_t ((u_t - v_t)/l_t)^2)
 *   K = [k(x_i,x_j)] + eta I;  L = chol(K);  alpha = K^{-1} y_k.
 * The factorisation runs in fp64 on the device. The model keeps alpha
 * (fp32), the lengthscale-scaled X and L^{-1} as the scoring kernel's
 * operand: the lower 16x32 blocks, each 16-row block scaled by a power of two
 * that puts its largest entry in [2^13, 2^14), every entry split into two
 * fp16 halves (hi = fp16(w), lo = fp16(w - hi)). It also extracts the
 * non-dominated set of Y on the host.
 *
 * Precision of the scores (fp32-class). The posterior runs in fp32 with the
 * triangular product on the fp16 matrix cores as three split products with
 * fp32 accumulation; both of its operands are scaled by powers of two first
 * (the candidates' kernel values per candidate, L^{-1} per row block), so
 * no value can overflow fp16 and each carries 22 significant bits (an
 * absolute floor of 2^-39 of its block's largest), against 24 in fp32. The
 * error of mu, of sigma^2 relative to the prior variance and of the EHVI is
 * therefore that of an fp32 implementation up to a small factor, for every
 * accepted hyperparameter. Where the posterior variance is far below the
 * prior (candidates near the data, long learned lengthscales) fp32 itself
 * loses sigma's relative accuracy: sigma^2 = k(x,x) - |v|^2 cancels.
 *
 * Accepted hyperparameters: outputscale in [2^-64, 2^64], noise in
 * [0, 2^64]. The model is refused with ILL_CONDITIONED when, for some
 * objective, max_i K_ii * max |L^{-1}|^2 (a lower bound on cond(K)) reaches
 * 2^24, where no fp32 solve carries a correct bit (e.g. near-duplicate
 * observations with zero noise).
 *
 * X      device [n][d]   encoded observations
 * Y      device [n][m]   standardised objective values (maximise)
 * n      1..BO_MAX_N;  d 1..BO_MAX_D;  m in {2, 3}
 * lengthscale host [m][d] > 0;  outputscale host [m] > 0;  noise host [m] >= 0
 * stream hipStream_t or NULL
 * out    receives a new model on BO_OK (untouched otherwise)
 *
 * Synchronous: enqueues all device work on the stream (behind earlier work,
 * without waiting for it), then waits once and returns after the positive
 * definiteness flag, the conditioning estimate and Y have been read back. Y
 * lives on the device, so its finiteness is checked once it is back (it is
 * read back first, so the host checks it and forms its front while the
 * device factors; the kernels run either way); the host arguments are
 * validated before anything is enqueued. Part of the work (the Gram matrix
 * past its first 64 columns, the scaled X and its distance fragments) runs
 * on a second stream of the library's own, at default priority, ordered
 * after the caller's earlier work and joined back into the caller's stream
 * once the factorisation is done (alpha and the packing follow there). Concurrent fits on one
 * device share a pinned staging buffer and run one at a time.
 * Memory: the model's device buffers are one allocation from a stream-ordered
 * pool (bo_free keeps the largest released one per device, once no work on it
 * is pending, and the next fit reuses it when it is large enough); the fp64
 * factorisation scratch (2 m n_f^2 doubles with n_f the
 * multiple of 64 at or above n, plus a few KB) is kept per device after the
 * first fit and reused, growing when a larger fit needs more (at most 201 MB,
 * at n = 2048, m = 3), until the process ends.
 * Errors: INVALID_ARGUMENT (also hyperparameters outside the accepted
 * range), NONFINITE_INPUT (hyperparameters or Y not finite), CAPACITY,
 * NOT_POSITIVE_DEFINITE (a pivot <= 0 or a non-finite inverse factor),
 * ILL_CONDITIONED, OUT_OF_MEMORY, DEVICE.
 */
bo_status bo_fit(const float* X, const float* Y, int64_t n, int32_t d, int32_t m,
                 const float* lengthscale, const float* outputscale,
                 const float* noise, void* stream, bo_model* out);

/*
 * bo_fit_composite — bo_fit with the paper's composite surrogate kernel.
 *
 * Paper: paragraphs "Additive kernels" and S5 "Model-GPU preference
 * encoding" of the online phase, and the kernel list of the implementation
 * section (ARD Matern-5/2 on the routing features, ARD Matern-3/2 on the
 * deployment features wrapped in the preference-weighted kernel, their
 * product as a low-weight interaction, each in its own scale kernel).
 *
 * With x = (tau, c): tau the first d_route coordinates (routing), c the
 * other d - d_route (deployment), and for objective k
 *   k(x, x') = s_route[k] M52(r_tau) + s_dep[k] w(c) w(c') M32(r_c)
 *              + s_int[k] M52(r_tau) M32(r_c),
 *   M52(r) = (1 + sqrt5 r + 5/3 r^2) exp(-sqrt5 r),
 *   M32(r) = (1 + sqrt3 r) exp(-sqrt3 r),
 *   r_tau, r_c the lengthscale-scaled distances over the two groups,
 *   w(c) = exp(sum_j pref[k][j] c_j)   (pref[k][j] = beta_k times the
 *          preference of the GPU type that deployment coordinate j counts).
 * The rest is as bo_fit: K = [k(x_i, x_j)] + eta I in fp64, L^{-1} and
 * alpha kept for scoring. The prior variance of a point is
 * s_route + s_dep w(c)^2 + s_int.
 *
 * d_route     1 <= d_route < d; the padded routing and deployment groups
 *             (each rounded up to a multiple of 4) must fit BO_MAX_D
 * lengthscale host [m][d] > 0 (routing then deployment coordinates)
 * scale_route host [m] > 0;  scale_dep, scale_int host [m] >= 0
 * pref        host [m][d - d_route], finite
 * Other arguments, behaviour and errors as bo_fit (CAPACITY when the padded
 * groups exceed BO_MAX_D). Models fitted this way score single points and
 * q-batches through bo_score; the batch factor's pivot rule takes the sum
 * of the three scales as the prior scale. They are also accepted by
 * bo_nehvi_prepare / bo_score_nehvi.
 */
bo_status bo_fit_composite(const float* X, const float* Y, int64_t n, int32_t d, int32_t m,
                           int32_t d_route, const float* lengthscale,
                           const float* scale_route, const float* scale_dep,
                           const float* scale_int, const float* pref, const float* noise,
                           void* stream, bo_model* out);

/*
 * bo_fit_f64 / bo_fit_composite_f64 — bo_fit and bo_fit_composite for scoring
 * in double precision.
 *
 * Paper: implementation section (the GP kernels are executed in double
 * precision; the hyperparameters are learned by maximising the marginal
 * likelihood). The fit is the same fp64 factorisation; the model also keeps
 * L^{-1} as fp64 fragments of the fp64 matrix cores, alpha and the inverse
 * lengthscales in fp64, and bo_score / bo_score_constrained / bo_score_noalloc
 * then compute the posterior in fp64 (scaled differences from the fp32
 * inputs, kernel values, mu, V = L^{-1} K*^T with fp64 accumulation, sigma^2
 * and the q x q factor), rounding mu, sigma and the factor to fp32 for the
 * acquisition, which is unchanged. Use it where the posterior variance lies
 * far below the prior (long learned lengthscales, candidates near the data):
 * there sigma^2 = k(x,x) - |v|^2 cancels beyond what fp32 resolves. The
 * triangle runs at the fp64 matrix rate, roughly 10x the fp32-class time.
 *
 * Arguments, behaviour and errors as bo_fit / bo_fit_composite, except that
 * the conditioning limit of ILL_CONDITIONED is 2^50 instead of 2^24. The
 * noisy acquisition (bo_nehvi_prepare) refuses these models
 * (INVALID_ARGUMENT).
 */
bo_status bo_fit_f64(const float* X, const float* Y, int64_t n, int32_t d, int32_t m,
                     const float* lengthscale, const float* outputscale,
                     const float* noise, void* stream, bo_model* out);
bo_status bo_fit_composite_f64(const float* X, const float* Y, int64_t n, int32_t d, int32_t m,
                               int32_t d_route, const float* lengthscale,
                               const float* scale_route, const float* scale_dep,
                               const float* scale_int, const float* pref, const float* noise,
                               void* stream, bo_model* out);

/*
 * bo_mll — exact log marginal likelihood of each objective's GP and its
 * gradient, for fitting the hyperparameters.
 *
 * Paper: implementation section (the ARD lengthscales and the scales are
 * learned by maximising the GP marginal likelihood). The outer optimiser
 * runs on the host and calls this for each trial point.
 *
 * For objective k, with K = s M52 + eta I exactly as in bo_fit:
 *   value[k] = -1/2 y^T K^{-1} y - 1/2 log det K - n/2 log(2 pi)
 *   grad[k][j] = d value[k] / d theta_j,
 *     theta = (log l_1 .. log l_d, log s, log eta)
 *           = 1/2 tr((alpha alpha^T - K^{-1}) dK/dtheta_j),  alpha = K^{-1} y.
 * Everything runs in fp64 on the device: the Cholesky factor and L^{-1} as
 * in bo_fit, K^{-1} = L^{-T} L^{-1}, the log-determinant from the diagonal
 * of L, and the trace terms over all pairs of observations.
 *
 * X, Y, n, d, m, lengthscale, outputscale, noise: as bo_fit
 * value  host [m] out;  grad  host [m][d + 2] out (fp64)
 * Synchronous; no model is created; uses the device's kept fp64 scratch as
 * bo_fit does. Errors: as bo_fit (NOT_POSITIVE_DEFINITE when K is not
 * positive definite).
 */
bo_status bo_mll(const float* X, const float* Y, int64_t n, int32_t d, int32_t m,
                 const float* lengthscale, const float* outputscale, const float* noise,
                 void* stream, double* value, double* grad);

/*
 * bo_score — posterior plus Monte-Carlo (q)EHVI for M candidates.
 *
 * Paper: "Constrained qNEHVI" paragraph (expected HVI over samples of the
 * joint posterior, Monte-Carlo integration) without the feasibility factor
 * (bo_score_constrained adds it), against the fixed front of the
 * observations.
 *
 * Per candidate batch b (q points x_1..x_q) and objective k:
 *   mu_a = k(x_a, X) alpha_k;  v_a = L_k^{-1} k(X, x_a);
 *   Sigma[a,b] = k(x_a, x_b) - v_a^T v_b;  C_k = chol_psd(Sigma) (q > 1)
 *   y_s[a,k] = mu_a + sigma_a z_s[0,k]               (q = 1)
 *   y_s[a,k] = mu_a + sum_c C_k[a,c] z_s[c,k]        (q > 1)
 *   ehvi[b] = 1/S sum_s qHVI({y_s[a,:]}) , the hypervolume improvement of
 *   the batch over the front F = non-dominated observations strictly above
 *   ref_point, computed over a disjoint box decomposition of the region F
 *   does not dominate (inclusion-exclusion over the 2^q - 1 member subsets).
 * chol_psd: no jitter; a Schur pivot <= 1e-10 * outputscale zeroes that
 * column. sigma = sqrt(max(Sigma[a,a], 0)).
 *
 * model        from bo_fit (same device must be current)
 * cand         device [M][q][d]
 * M            >= 0 (0 is a no-op);  q in {1, 2, 4}
 * ref_point    host [m], finite
 * base_samples device [S][q][m], standard normal draws shared by all M
 * S            1..BO_MAX_S
 * ehvi         device [M] out
 * mu, sigma    device [M][q][m] out, or NULL to skip writing them
 * stream       hipStream_t or NULL
 *
 * Asynchronous: enqueues kernels and returns. The box decomposition is built
 * on the host when ref_point (or the model) changes and copied with the
 * stream. Errors: INVALID_ARGUMENT, NONFINITE_INPUT (ref_point), CAPACITY
 * (box count, S), OUT_OF_MEMORY (workspace growth), DEVICE.
 */
bo_status bo_score(bo_model model, const float* cand, int64_t M, int32_t q,
                   const float* ref_point, const float* base_samples, int32_t S,
                   float* ehvi, float* mu, float* sigma, void* stream);

/*
 * bo_score_constrained — bo_score with the feasibility factor.
 *
 * Paper: "Constrained qNEHVI" paragraph. The constraints bound the
 * objectives themselves (a latency cap L <= L_max, a quality floor
 * Q >= Q_min, written g_i <= 0), and the acquisition is the expectation of
 * HVI times the indicator that every constraint holds, over the same joint
 * posterior samples. On the maximised, standardised objectives each
 * constraint reads y_k >= feas_lower[k]:
 *   q = 1: ehvi[b] = 1/S sum_s HVI(y_s) * prod_k 1[y_s[k] >= feas_lower[k]]
 *   q > 1: a batch member counts only on the samples where it is feasible:
 *          each inclusion-exclusion term of a member subset J is multiplied
 *          by the product of its members' indicators (= the HVI of the
 *          feasible members).
 * A sample exactly on a threshold is feasible.
 *
 * feas_lower host [m]: per-objective lower bound in standardised units;
 *            -inf leaves that objective unconstrained, +inf makes every
 *            sample infeasible (ehvi = 0); NULL is exactly bo_score.
 * Other arguments, ownership and errors as bo_score; NONFINITE_INPUT also
 * for a NaN threshold.
 */
bo_status bo_score_constrained(bo_model model, const float* cand, int64_t M, int32_t q,
                               const float* ref_point, const float* feas_lower,
                               const float* base_samples, int32_t S, float* ehvi,
                               float* mu, float* sigma, void* stream);

/*
 * bo_score_noalloc — bo_score (mu and sigma not returned) that allocates
 * nothing, for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.
 *
 * The same kernels and results as bo_score with mu = sigma = NULL (bitwise),
 * but the boxes and the posterior workspace live in a fixed 32 MiB device
 * array that the library holds on every device it runs on until the process
 * ends; no hipMalloc, hipFree, pinned host allocation or other allocating
 * library routine is called. Limit: M * q * m * 2 floats of workspace, plus
 * M * m * q(q+1)/2 for q > 1, must fit 32 MiB less the boxes' 96 KiB
 * (2,091,008 single points of two objectives; 154,889 q = 4 batches of three),
 * else CAPACITY before any device work.
 *
 * Every call on a device shares that device's array. Calls ordered on one
 * stream are safe (the box upload is stream-ordered behind the previous
 * call's kernels); calls that overlap on one device (different streams, or
 * threads) race on it and must be ordered by the caller. Nothing in the
 * array needs clearing: every call writes all of what it reads. The box
 * decomposition is rebuilt on the host and copied from pageable memory on
 * every call (that copy completes before the call returns).
 *
 * Arguments, asynchrony and errors: as bo_score (CAPACITY also for the limit
 * above).
 */
bo_status bo_score_noalloc(bo_model model, const float* cand, int64_t M, int32_t q,
                           const float* ref_point, const float* base_samples, int32_t S,
                           float* ehvi, void* stream);

/*
 * bo_nehvi_prepare / bo_score_nehvi — the noisy acquisition (qNEHVI;
 * candidates or q-batches, two or three objectives, Matern-5/2 or
 * composite-kernel models).
 *
 * Paper: workflow step (ii) and the "Constrained qNEHVI" paragraph (after
 * Daulton et al. 2021). The observations are noisy, so the latent objective
 * values at the observed points X are sampled too: draw s takes the latent f
 * jointly at X and at the batch B from the GP posterior, by the lower
 * Cholesky factor of the joint covariance applied to (z_X^s, z*^s):
 *   f_X^s = mu_X + L_XX z_X^s            (Sigma_XX = L_XX L_XX^T),
 *   f_B^s = E[f_B | f_X^s] + C z*^s,
 *   E[f_B | f_X] = K_BX K_XX^{-1} f_X,  C C^T = k(B,B) - K_BX K_XX^{-1} K_XB
 *   (K_XX the noise-free Gram matrix; the noisy y adds nothing once f_X is
 *   known; C by the PSD rule of bo_score's batch factor), and
 *   ehvi[b] = 1/S sum_s HVI_s(f_B^s),
 * where HVI_s is the joint hypervolume improvement of the members over the
 * Pareto front of the in-sample values f_X^s (maximise, strictly above
 * ref_point). With feasibility thresholds only the in-sample vectors meeting
 * all of them form the fronts, and a member counts only on the draws where it
 * is feasible (as in bo_score_constrained).
 *
 * bo_nehvi_prepare(model, base_samples_X, S, ref_point, feas_lower, stream):
 *   base_samples_X device [S][n][m] iid N(0,1), row-major (draw, observed
 *                  point, objective); 1 <= S <= 512
 *   ref_point      host [m];  feas_lower host [m] or NULL
 *   Builds, in fp64 on the device, the in-sample posterior and its factor,
 *   the S in-sample draws, each draw's front and box decomposition, the
 *   factor of K_XX (on a library-owned second stream of the model's device,
 *   joined back to `stream`) and G = K_XX^{-1} L_XX Z_X; keeps them in the
 *   model (replacing an earlier preparation). Synchronous.
 *   Errors: INVALID_ARGUMENT (m not 2 or 3, bad S or pointer), CAPACITY (S > 512, too many boxes), NOT_POSITIVE_DEFINITE (K,
 *   the in-sample covariance or K_XX), NONFINITE_INPUT, OUT_OF_MEMORY,
 *   DEVICE.
 *
 * bo_score_nehvi(model, cand, M, q, base_samples, S, ehvi, stream):
 *   cand device [M][q][d] (q in {1, 2, 4}); base_samples device [S][q][m]
 *   (z*, shared by all batches); S must equal the prepared S; ehvi device [M]
 *   out. Asynchronous; batches are processed in chunks of 1048576 points,
 *   whose per-draw conditional means (m x S x chunk floats) live in a
 *   model-owned workspace that grows on first use.
 *   Errors: INVALID_ARGUMENT (not prepared, S mismatch, bad q, pointers),
 *   CAPACITY, OUT_OF_MEMORY, DEVICE.
 *
 * bo_nehvi_front(model, sample, idx_host, cap, count): the front of one
 *   draw (indices into the observations, sorted by objective 0 ascending),
 *   min(cap, size) entries to host memory, *count = its size. Synchronous.
 */
bo_status bo_nehvi_prepare(bo_model model, const float* base_samples_X, int32_t S,
                           const float* ref_point, const float* feas_lower, void* stream);
bo_status bo_score_nehvi(bo_model model, const float* cand, int64_t M, int32_t q,
                         const float* base_samples, int32_t S, float* ehvi, void* stream);
bo_status bo_nehvi_front(bo_model model, int32_t sample, int32_t* idx_host, int32_t cap,
                         int32_t* count);

/*
 * bo_argmax — first index of the maximum of values[0..M).
 *
 * Paper: workflow step (ii), choosing theta* as the maximiser of the
 * acquisition over the candidates.
 *
 * values device [M];  M in [0, 2^31)
 * index  device int64 out: lowest index among equal maxima; NaN never wins;
 *        -1 when M == 0 or every value is NaN
 * value  device float out: values[index], or NaN when index == -1
 * Asynchronous. Uses *index as its own reduction cell (no workspace).
 * Errors: INVALID_ARGUMENT.
 */
bo_status bo_argmax(const float* values, int64_t M, int64_t* index, float* value,
                    void* stream);

/* Number of non-dominated observations kept by bo_fit (before the
 * reference-point filter), or -1 for a NULL model. */
int32_t bo_model_front_size(bo_model model);

/* Copies min(cap, front size) indices (into Y rows) of the non-dominated
 * observations, sorted by objective 0 ascending then index, to host memory.
 * Errors: INVALID_ARGUMENT. */
bo_status bo_model_front_indices(bo_model model, int32_t* idx_host, int32_t cap);

/*
 * bo_cholesky_test — the blocked right-looking Cholesky used by bo_fit,
 * exposed so its failure path can be tested.
 * A device [n][n] symmetric (lower triangle read), L device [n][n] out
 * (lower factor, zeros above the diagonal). 1 <= n <= BO_MAX_N.
 * Synchronous. Errors: INVALID_ARGUMENT, NOT_POSITIVE_DEFINITE (a pivot
 * <= 0 or non-finite), OUT_OF_MEMORY, DEVICE.
 */
bo_status bo_cholesky_test(const float* A, int64_t n, float* L, void* stream);

/*
 * bo_draw_fronts3_test — the per-draw fronts and box decompositions that
 * bo_nehvi_prepare builds for three objectives, exposed so their rules can be
 * tested on chosen values (ties, duplicates, thresholds).
 * Paper: "Constrained qNEHVI" paragraph (each sample's improvement is
 * measured against the Pareto front of that sample's in-sample values).
 * F      device [S][n][3] fp64 values (draw, point, objective)
 * ref    host [3]; feas_lower host [3] or NULL (rows failing any threshold
 *        take no part)
 * front  device [S][n] int32 out: per draw, its first P entries are the
 *        front's indices (non-dominated among the points strictly above ref,
 *        exact duplicates keep the lowest index), objective 0 ascending then
 *        index; the rest is unspecified
 * boxes  device [S][3n + 1][6] fp32 out: per draw, its first counts[s] boxes
 *        (lo0, lo1, lo2, w0, w1, w2), disjoint, covering the part of the
 *        region above ref that the front does not dominate (inf widths for
 *        unbounded sides)
 * counts device [2S] int32 out: the number of boxes per draw, then P
 * 1 <= n <= BO_MAX_N, S >= 1. Synchronous.
 * Errors: INVALID_ARGUMENT, CAPACITY, NONFINITE_INPUT (ref, a NaN threshold,
 * or a non-finite value of F), OUT_OF_MEMORY, DEVICE.
 */
bo_status bo_draw_fronts3_test(const double* F, int64_t n, int32_t S, const float* ref,
                               const float* feas_lower, int32_t* front, float* boxes,
                               int32_t* counts, void* stream);

/*
 * Host-only geometry (no device work; callable without a GPU).
 *
 * bo_pareto_front: non-dominated rows of Y (maximise; duplicates keep the
 * lowest index) that are strictly above ref in every objective, sorted by
 * objective 0 ascending then index. Y host [n][m], ref host [m] or NULL
 * (no reference filter). Writes min(cap, count) indices; *count gets the
 * full count.
 *
 * bo_box_decomposition: disjoint boxes [lo, hi) covering
 * {z > ref : no f in F with f >= z} for a front F host [P][m] (m in {2,3},
 * every row strictly above ref). hi may be +inf. lo/hi host [cap][m];
 * *count gets the number of boxes (BO_ERR_CAPACITY when it exceeds cap).
 */
bo_status bo_pareto_front(const float* Y, int64_t n, int32_t m, const float* ref,
                          int32_t* idx, int32_t cap, int32_t* count);
bo_status bo_box_decomposition(const float* F, int32_t P, int32_t m,
                               const float* ref, float* lo, float* hi,
                               int32_t cap, int32_t* count);

/*
 * Phase timing for benchmarks. While enabled, every bo_score call records
 * HIP events on its stream before its posterior launches, between them and
 * the (q)EHVI launch, and after it. bo_profile_read waits for the recorded
 * events, returns the summed milliseconds of each phase, the number of
 * bo_score calls and the number of posterior launches (one per objective per
 * call) since the last read, and clears them. Enabling resets the counters.
 * Up to 4096 calls are kept; later calls are not timed (see *calls).
 * Errors: INVALID_ARGUMENT (NULL output), DEVICE.
 */
bo_status bo_profile_enable(int32_t on);
bo_status bo_profile_read(double* posterior_ms, double* ehvi_ms, int64_t* calls,
                          int64_t* posterior_launches);

/*
 * Device characterisation for roofline fractions: runs a fixed synthetic
 * workload over the whole chip on `stream`, synchronously, and returns the
 * achieved rate in *rate:
 *   BO_PEAK_VALU_FMA   lane-ops/s of independent fp32 FMA chains (no packed math)
 *   BO_PEAK_VALU_CLAMP lane-ops/s of the (sub, med3, fma) pattern of the EHVI loop
 *   BO_PEAK_MFMA_F32   flop/s of independent v_mfma_f32_16x16x4f32 chains
 *   BO_PEAK_HBM_COPY   bytes/s (read + write) of a 1 GiB streaming copy
 *   BO_PEAK_MFMA_F16   flop/s of independent v_mfma_f32_16x16x32_f16 chains
 * iters: inner iterations for the compute probes (ignored by the copy).
 * Allocates its own buffers. Errors: INVALID_ARGUMENT, DEVICE, OUT_OF_MEMORY.
 */
#define BO_PEAK_VALU_FMA 0
#define BO_PEAK_VALU_CLAMP 1
#define BO_PEAK_MFMA_F32 2
#define BO_PEAK_HBM_COPY 3
#define BO_PEAK_MFMA_F16 4
bo_status bo_measure_peak(int32_t what, int64_t iters, double* rate, void* stream);

/* Releases a model (waits for its last stream first). NULL is a no-op. */
void bo_free(bo_model model);

/* Static description of a status code. */
const char* bo_status_string(bo_status status);

/* Detail of the last error on the calling thread ("" if none). */
const char* bo_last_error_message(void);

#ifdef __cplusplus
}
#endif

#endif /* BO_H_ */
