// C ABI entry points: validation, model lifecycle and launch sequencing.
//
// bo_fit      — Gram (fp64) -> blocked Cholesky -> L^{-1} -> alpha -> pack,
//               all on the caller's stream, then one synchronisation to read
//               the positive-definiteness flag back.
// bo_score    — per objective one posterior launch, then one (q)EHVI launch
//               (bo_score_constrained: the same with feasibility weights);
//               asynchronous. The box decomposition is rebuilt on the host
//               only when the reference point changes.
// bo_argmax   — three tiny launches using the caller's index cell.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "bo_internal.h"

namespace bo {

size_t posterior_lds_bytes(int nb, int q);
size_t ehvi_lds_bytes(int S, int q, int m, int nbox);

namespace {
thread_local std::string g_err;

bool sync_debug() {
  static int v = [] {
    const char* e = std::getenv("BO_SYNC_DEBUG");
    return (e && e[0] == '1') ? 1 : 0;
  }();
  return v != 0;
}

constexpr size_t kLdsLimit = 160 * 1024;

// Device pointer check: the whole [p, p + bytes) must lie in one device
// allocation of the current device.
bo_status check_dev(const void* p, size_t bytes, const char* name) {
  if (!p) return fail(BO_ERR_INVALID_ARGUMENT, std::string(name) + " is NULL");
  hipPointerAttribute_t attr;
  hipError_t e = hipPointerGetAttributes(&attr, p);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(BO_ERR_INVALID_ARGUMENT, std::string(name) + " is not a device pointer");
  }
  if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged) {
    return fail(BO_ERR_INVALID_ARGUMENT, std::string(name) + " is not device memory");
  }
  int dev = -1;
  (void)hipGetDevice(&dev);
  if (attr.device != dev) {
    return fail(BO_ERR_INVALID_ARGUMENT, std::string(name) + " lives on another device");
  }
  if (bytes > 0) {
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    e = hipMemGetAddressRange(&base, &size, const_cast<void*>(p));
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(BO_ERR_INVALID_ARGUMENT, std::string(name) + ": no allocation range");
    }
    const char* b = static_cast<const char*>(base);
    const char* q = static_cast<const char*>(p);
    if (q < b || static_cast<size_t>(q - b) + bytes > size) {
      return fail(BO_ERR_INVALID_ARGUMENT,
                  std::string(name) + " is smaller than the sizes passed require");
    }
  }
  return BO_OK;
}

bo_status after_launch(hipError_t e, hipStream_t st, const char* what) {
  if (e != hipSuccess) return hip_fail(e, what);
  if (sync_debug()) {
    e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, what);
  }
  return BO_OK;
}


bool all_finite(const float* v, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!std::isfinite(v[i])) return false;
  return true;
}

// Per-device library state: a stream-ordered memory pool (allocations made
// and released inside the hot path come back from it without a device-wide
// synchronisation), one pinned staging buffer for box uploads, and one for
// the fit's uploads and read-backs (pinned, so that bo_fit enqueues all of its
// work without waiting for earlier work on the stream; bo_fit holds fit_mu
// until its final synchronisation, so the buffer is never rewritten while a
// copy from it is pending).
struct DeviceState {
  std::mutex mu;
  hipMemPool_t pool = nullptr;
  // under mu: one released model allocation kept for the next fit (nothing
  // pending on it), so a fit-score-release loop neither frees nor allocates
  unsigned char* spare = nullptr;
  size_t spare_bytes = 0;
  float* stage = nullptr;
  size_t stage_floats = 0;
  hipEvent_t stage_evt = nullptr;
  std::mutex fit_mu;
  unsigned char* fit_stage = nullptr;
  size_t fit_stage_bytes = 0;
  // under fit_mu: a second stream (default priority) for independent work
  // inside one call, joined back by the two events
  hipStream_t side = nullptr;
  hipEvent_t side_evt[3] = {nullptr, nullptr, nullptr};
  // under fit_mu: the fp64 scratch of bo_fit and bo_mll, kept and grown on
  // demand (both synchronise their stream before releasing fit_mu, so none
  // of it is in use between calls): A, W [mat], hyperparameters [nhyp],
  // vector [vec], hyperparameters [nhyp], then 64 bytes of flag (int) and
  // statistics (at byte 16), then the row-block maxima [3][BO_MAX_N / 16]
  // (kFitSmall bytes in all)
  double* fw = nullptr;
  size_t fw_mat = 0, fw_hyp = 0, fw_vec = 0;
  // under fit_mu: marks bo_fit's early read-back of Y
  hipEvent_t fit_evt = nullptr;
};

// The side stream and its events of device state DS (created once).
bo_status side_stream(DeviceState* DS) {
  if (DS->side) return BO_OK;
  hipError_t e = hipStreamCreateWithFlags(&DS->side, hipStreamNonBlocking);
  if (e != hipSuccess) { DS->side = nullptr; return hip_fail(e, "side stream"); }
  for (int i = 0; i < 3; ++i) {
    e = hipEventCreateWithFlags(&DS->side_evt[i], hipEventDisableTiming);
    if (e != hipSuccess) return hip_fail(e, "side stream event");
  }
  return BO_OK;
}
constexpr int kMaxDevices = 64;

DeviceState* device_state(int dev) {
  static DeviceState states[kMaxDevices];
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  return &states[dev];
}

bo_status get_pool(int dev, hipMemPool_t* out) {
  DeviceState* S = device_state(dev);
  if (!S) return fail(BO_ERR_DEVICE, "device index out of range");
  std::lock_guard<std::mutex> lk(S->mu);
  if (!S->pool) {
    hipMemPoolProps props = {};
    props.allocType = hipMemAllocationTypePinned;
    props.location.type = hipMemLocationTypeDevice;
    props.location.id = dev;
    hipError_t e = hipMemPoolCreate(&S->pool, &props);
    if (e != hipSuccess) { S->pool = nullptr; return hip_fail(e, "hipMemPoolCreate"); }
    uint64_t keep = UINT64_MAX;      // never trim: reuse across calls
    e = hipMemPoolSetAttribute(S->pool, hipMemPoolAttrReleaseThreshold, &keep);
    if (e != hipSuccess) return hip_fail(e, "hipMemPoolSetAttribute");
  }
  *out = S->pool;
  return BO_OK;
}

// Stream-ordered allocation of `count` elements on the current device.
template <typename T>
bo_status palloc(T** p, size_t count, hipStream_t st, const char* what) {
  *p = nullptr;
  if (count == 0) return BO_OK;
  int dev = 0;
  (void)hipGetDevice(&dev);
  hipMemPool_t pool;
  bo_status s = get_pool(dev, &pool);
  if (s != BO_OK) return s;
  void* q = nullptr;
  hipError_t e = hipMallocFromPoolAsync(&q, sizeof(T) * count, pool, st);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(BO_ERR_OUT_OF_MEMORY, std::string("device allocation failed for ") + what);
  }
  *p = static_cast<T*>(q);
  return BO_OK;
}

template <typename T>
void pfree(T*& p, hipStream_t st) {
  if (p) (void)hipFreeAsync(p, st);
  p = nullptr;
}

struct DeviceGuard {
  int prev = -1;
  bool ok = true;
  explicit DeviceGuard(int dev) {
    (void)hipGetDevice(&prev);
    if (prev != dev) ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    int cur = -1;
    (void)hipGetDevice(&cur);
    if (prev >= 0 && cur != prev) (void)hipSetDevice(prev);
  }
};

// Temporary device buffers of the fit, returned to the pool on every exit
// path (ordered after the fit's work on its stream).
// fp64 fit scratch: the device's kept workspace (fit_work), or buffers of
// its own (own = true, freed on destruction).
struct FitScratch {
  hipStream_t st = nullptr;
  bool own = false;
  double* A = nullptr;
  double* W = nullptr;
  double* hyp = nullptr;
  double* tmp = nullptr;
  int* flag = nullptr;
  unsigned long long* stats = nullptr;   // [2m]: max K_ii, then max |L^{-1}| (double bits)
  unsigned long long* bmax = nullptr;    // [m][nb]: row-block maxima of |L^{-1}| (kept scratch)
  size_t hyp_cap = 0;                    // kept scratch: doubles from hyp to flag
  ~FitScratch() {
    if (!own) return;
    pfree(A, st); pfree(W, st); pfree(hyp, st); pfree(tmp, st); pfree(flag, st);
    pfree(stats, st);
  }
};

// Releases the device buffers of a model after all device work (not the host
// object). The caller may have used the model on several streams, so wait
// for the whole device before handing memory back to the pool.
void release_noisy(Model* M) {
  Model::Noisy& z = M->nz;
  if (z.Lp0 || z.Gp || z.boxes || z.off || z.front || z.ws) (void)hipDeviceSynchronize();
  pfree(z.Lp0, nullptr);
  pfree(z.Gp, nullptr);
  pfree(z.boxes, nullptr);
  pfree(z.off, nullptr);
  pfree(z.front, nullptr);
  pfree(z.ws, nullptr);
  z.ws_floats = 0;
  z.S = z.Sp = z.n32 = z.total = 0;
  z.counts.clear();
  z.fsize.clear();
}

void release_buffers(Model* M) {
  release_noisy(M);
  if ((M->arena && M->pending) || M->ws || M->d_boxes) (void)hipDeviceSynchronize();
  if (M->arena) {
    // nothing reads the allocation any more: keep the larger of it and the
    // device's spare for the next fit, free the other
    DeviceState* DS = device_state(M->device);
    unsigned char* drop = M->arena;
    if (DS) {
      std::lock_guard<std::mutex> lk(DS->mu);
      if (M->arena_bytes > DS->spare_bytes) {
        drop = DS->spare;
        DS->spare = M->arena;
        DS->spare_bytes = M->arena_bytes;
      }
    }
    pfree(drop, nullptr);
    M->arena = nullptr;
    M->arena_bytes = 0;
  }
  M->Lp64 = nullptr; M->alpha64 = nullptr; M->ils64 = nullptr;
  M->xf = nullptr; M->x2 = nullptr; M->ctr = nullptr; M->Xd = nullptr;
  M->Xs = nullptr; M->invls = nullptr; M->alpha = nullptr; M->Lp = nullptr;
  M->wts = nullptr; M->pref = nullptr;
  pfree(M->ws, nullptr);
  pfree(M->d_boxes, nullptr);
}

// Bytes after the fit scratch's vector: flag and statistics (64), then the
// row-block maxima of |L^{-1}| for up to three objectives.
constexpr size_t kFitSmall = 64 + sizeof(unsigned long long) * 3 * (BO_MAX_N / kBlk);

// The device's kept fit scratch, grown to at least the given sizes (the
// caller holds DS->fit_mu). Growing waits for the device, then replaces the
// buffer.
bo_status fit_work(DeviceState* DS, size_t mat, size_t nhyp, size_t vec, FitScratch* fs) {
  if (!DS->fw || mat > DS->fw_mat || nhyp > DS->fw_hyp || vec > DS->fw_vec) {
    const size_t m2 = std::max(mat, DS->fw_mat), h2 = std::max(nhyp, DS->fw_hyp),
                 v2 = std::max(vec, DS->fw_vec);
    if (DS->fw) {
      (void)hipDeviceSynchronize();
      (void)hipFree(DS->fw);
      DS->fw = nullptr;
      DS->fw_mat = DS->fw_hyp = DS->fw_vec = 0;
    }
    void* q = nullptr;
    hipError_t e = hipMalloc(&q, sizeof(double) * (2 * m2 + h2 + v2) + kFitSmall);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(BO_ERR_OUT_OF_MEMORY, "device allocation failed for the fit scratch");
    }
    DS->fw = static_cast<double*>(q);
    DS->fw_mat = m2; DS->fw_hyp = h2; DS->fw_vec = v2;
  }
  // [A][W][vector][hyperparameters][flag, statistics, maxima]: the last two
  // are contiguous, so one upload sets both
  fs->own = false;
  fs->A = DS->fw;
  fs->W = fs->A + DS->fw_mat;
  fs->tmp = fs->W + DS->fw_mat;
  fs->hyp = fs->tmp + DS->fw_vec;
  fs->hyp_cap = DS->fw_hyp;
  fs->flag = reinterpret_cast<int*>(fs->hyp + DS->fw_hyp);
  fs->stats = reinterpret_cast<unsigned long long*>(fs->hyp + DS->fw_hyp + 2);
  fs->bmax = reinterpret_cast<unsigned long long*>(fs->hyp + DS->fw_hyp + 8);
  return BO_OK;
}

// Byte offsets of a model's buffers inside its arena (256-byte aligned).
struct ArenaLayout {
  size_t total = 0;
  size_t add(size_t bytes) {
    const size_t o = total;
    total += (bytes + 255) / 256 * 256;
    return o;
  }
};

// Phase timing (bo_profile_enable / bo_profile_read).
struct Profile {
  std::mutex mu;
  bool on = false;
  struct Rec { hipEvent_t e[3]; int launches; };
  std::vector<Rec> pool;
  size_t used = 0;
};
Profile& profile() {
  static Profile p;
  return p;
}
constexpr size_t kProfileCap = 4096;

}  // namespace

bo_status fail(bo_status st, const std::string& msg) {
  g_err = msg;
  return st;
}

bo_status hip_fail(hipError_t e, const char* what) {
  g_err = std::string(what) + ": " + hipGetErrorString(e);
  (void)hipGetLastError();
  return (e == hipErrorOutOfMemory) ? BO_ERR_OUT_OF_MEMORY : BO_ERR_DEVICE;
}

}  // namespace bo

struct bo_model_s {
  bo::Model m;
};

using namespace bo;

extern "C" {

const char* bo_status_string(bo_status s) {
  switch (s) {
    case BO_OK: return "ok";
    case BO_ERR_INVALID_ARGUMENT: return "invalid argument";
    case BO_ERR_NOT_POSITIVE_DEFINITE: return "matrix not positive definite";
    case BO_ERR_CAPACITY: return "size beyond compiled capacity";
    case BO_ERR_DEVICE: return "HIP runtime error";
    case BO_ERR_OUT_OF_MEMORY: return "out of memory";
    case BO_ERR_NONFINITE_INPUT: return "non-finite input";
    case BO_ERR_ILL_CONDITIONED: return "covariance too ill-conditioned for fp32-class scoring";
  }
  return "unknown status";
}

const char* bo_last_error_message(void) { return g_err.c_str(); }

bo_status bo_pareto_front(const float* Y, int64_t n, int32_t m, const float* ref,
                          int32_t* idx, int32_t cap, int32_t* count) {
  if (!Y || !count || (cap > 0 && !idx) || n < 0 || cap < 0)
    return fail(BO_ERR_INVALID_ARGUMENT, "bo_pareto_front: bad pointer or size");
  if (m < 1 || m > 8) return fail(BO_ERR_INVALID_ARGUMENT, "bo_pareto_front: m out of range");
  std::vector<int32_t> out;
  host_front(Y, n, m, ref, out);
  *count = static_cast<int32_t>(out.size());
  const int32_t k = std::min<int32_t>(cap, *count);
  for (int32_t i = 0; i < k; ++i) idx[i] = out[i];
  return BO_OK;
}

bo_status bo_box_decomposition(const float* F, int32_t P, int32_t m, const float* ref,
                               float* lo, float* hi, int32_t cap, int32_t* count) {
  if ((P > 0 && !F) || !ref || !count || P < 0 || cap < 0 || (cap > 0 && (!lo || !hi)))
    return fail(BO_ERR_INVALID_ARGUMENT, "bo_box_decomposition: bad pointer or size");
  if (m != 2 && m != 3) return fail(BO_ERR_INVALID_ARGUMENT, "bo_box_decomposition: m must be 2 or 3");
  if (!all_finite(ref, m) || !all_finite(F, static_cast<size_t>(P) * m))
    return fail(BO_ERR_NONFINITE_INPUT, "bo_box_decomposition: non-finite input");
  for (int32_t i = 0; i < P; ++i)
    for (int k = 0; k < m; ++k)
      if (!(F[i * m + k] > ref[k]))
        return fail(BO_ERR_INVALID_ARGUMENT, "bo_box_decomposition: front row not above ref");
  std::vector<float> Fs;
  const float* Fp = F;
  if (m == 2) {
    // the staircase needs the 2-D non-dominated points sorted by objective 0
    std::vector<int32_t> nd;
    host_front<float>(F, P, 2, nullptr, nd);
    for (int32_t i : nd) { Fs.push_back(F[2 * i]); Fs.push_back(F[2 * i + 1]); }
    Fp = Fs.data();
    P = static_cast<int32_t>(nd.size());
  }
  std::vector<float> l, h;
  host_boxes(Fp, P, m, ref, l, h);
  const int32_t nbx = static_cast<int32_t>(l.size() / m);
  *count = nbx;
  if (nbx > cap) return fail(BO_ERR_CAPACITY, "bo_box_decomposition: cap too small");
  std::memcpy(lo, l.data(), sizeof(float) * l.size());
  std::memcpy(hi, h.data(), sizeof(float) * h.size());
  return BO_OK;
}

int32_t bo_model_front_size(bo_model model) {
  if (!model) return -1;
  return static_cast<int32_t>(model->m.nd.size());
}

bo_status bo_model_front_indices(bo_model model, int32_t* idx_host, int32_t cap) {
  if (!model || (cap > 0 && !idx_host) || cap < 0)
    return fail(BO_ERR_INVALID_ARGUMENT, "bo_model_front_indices: bad argument");
  const int32_t k = std::min<int32_t>(cap, static_cast<int32_t>(model->m.nd.size()));
  for (int32_t i = 0; i < k; ++i) idx_host[i] = model->m.nd[i];
  return BO_OK;
}

}  // extern "C"

namespace {

// Composite-kernel hyperparameters as passed to bo_fit_composite (host).
// Accepted hyperparameter range: output scales in [2^-64, 2^64], noise and
// the composite's other scales in [0, 2^64]. Inside it every intermediate of
// the fp32 scoring arithmetic (scaled squared norms, variances) stays in
// fp32's normal range.
constexpr double kScaleMin = 0x1p-64, kScaleMax = 0x1p64;
// A fitted model is refused (BO_ERR_ILL_CONDITIONED) when max K_ii times
// max |L^{-1}|^2, a lower bound on the condition number of K, reaches 2^24:
// beyond it the fp32-class solve, like any fp32 one, carries no correct bit.
constexpr double kCondLimit = 0x1p24;
// The same estimate's limit for fp64 scoring (bo_fit_f64): 2^50.
constexpr double kCondLimitF64 = 0x1p50;

double bits_to_double(unsigned long long b) {
  double v;
  std::memcpy(&v, &b, sizeof(v));
  return v;
}

// Calls on one model may come on different streams. Each scoring call first
// makes its stream wait for the model's previous call (when that ran on
// another stream) and records an event at its end, so a call never rewrites
// the boxes or the workspace while an earlier call may still read them.
bo_status order_after_previous(Model& M, hipStream_t st, const char* who) {
  M.pending = true;
  if (M.last_evt && M.last_stream != st) {
    hipError_t e = hipStreamWaitEvent(st, M.last_evt, 0);
    if (e != hipSuccess) return hip_fail(e, who);
  }
  return BO_OK;
}
bo_status mark_call(Model& M, hipStream_t st, const char* who) {
  M.pending = true;
  if (!M.last_evt) {
    hipError_t e = hipEventCreateWithFlags(&M.last_evt, hipEventDisableTiming);
    if (e != hipSuccess) {
      M.last_evt = nullptr;
      return hip_fail(e, who);
    }
  }
  hipError_t e = hipEventRecord(M.last_evt, st);
  if (e != hipSuccess) return hip_fail(e, who);
  M.last_stream = st;
  return BO_OK;
}

// Arguments of the posterior kernel for objective k of a fitted model: the
// packed inverse factor Lp (the model's, or the noisy acquisition's noise-free
// one, its row-block scales after its fragments); outputs are the caller's to
// set.
PosteriorArgs posterior_args(const Model& M, int k, const float* Lp,
                             const float* cand, int64_t npts, int q) {
  PosteriorArgs pa;
  pa.cand = cand; pa.npts = npts; pa.d = M.d; pa.dx = M.dx; pa.q = q;
  pa.Xs = M.Xs + (size_t)k * M.n_pad * M.dx;
  pa.invls = M.invls + (size_t)k * M.dx;
  pa.alpha = M.alpha + (size_t)k * M.n_pad;
  pa.Lp = Lp + (size_t)k * M.lp_per_obj;
  pa.kbound = M.kbound[k];
  {
    // a plain model's kernel values are at most s: scale them by 2^(14 - E)
    // for the split (the kernel multiplies s by it, exactly)
    int E = 0;
    (void)std::frexp(static_cast<double>(M.os[k]), &E);
    pa.ss = static_cast<float>(std::ldexp(static_cast<double>(M.os[k]), 14 - E));
    pa.kinv0 = static_cast<float>(std::ldexp(1.0, E - 14));
  }
  pa.xf = M.xf + (size_t)k * M.nb * dist_frags(M.dx) * 512;
  pa.x2 = M.x2 + (size_t)k * 2 * M.n_pad;
  pa.ctr = M.ctr + (size_t)k * M.dx;
  pa.n = static_cast<int>(M.n); pa.nb = M.nb;
  pa.s = M.os[k];
  pa.m = M.m; pa.k = k;
  pa.dr = M.dr; pa.dr4 = M.dr4;
  pa.s_dep = M.dr > 0 ? M.s_dep[k] : 0.f;
  pa.s_int = M.dr > 0 ? M.s_int[k] : 0.f;
  pa.wts = M.dr > 0 ? M.wts + (size_t)k * M.n_pad : nullptr;
  pa.pref = M.dr > 0 ? M.pref + (size_t)k * (M.d - M.dr) : nullptr;
  if (M.f64) {
    pa.Lp64 = M.Lp64 + (size_t)k * posterior_f64_blocks(M.nb) * 512;
    pa.alpha64 = M.alpha64 + (size_t)k * M.n_fit;
    pa.ils64 = M.ils64 + (size_t)k * M.d;
    pa.Xraw = M.Xd;
  }
  return pa;
}

// ---- scoring, shared by bo_score and the no-allocation variant ----------

// Host-side validation of a scoring call (nothing is enqueued).
bo_status score_validate(const char* who, bo_model model, const float* cand, int64_t M_,
                         int32_t q, const float* ref_point, const float* feas_lower,
                         const float* base_samples, int32_t S, float* ehvi, float* mu,
                         float* sigma) {
  (void)cand; (void)base_samples; (void)ehvi; (void)mu; (void)sigma;
  const std::string W(who);
  if (!model) return fail(BO_ERR_INVALID_ARGUMENT, W + ": model is NULL");
  Model& M = model->m;
  if (M_ < 0) return fail(BO_ERR_INVALID_ARGUMENT, W + ": M < 0");
  if (q != 1 && q != 2 && q != 4) return fail(BO_ERR_INVALID_ARGUMENT, W + ": q must be 1, 2 or 4");
  if (S < 1) return fail(BO_ERR_INVALID_ARGUMENT, W + ": S < 1");
  if (S > BO_MAX_S) return fail(BO_ERR_CAPACITY, W + ": S beyond compiled limit");
  if (!ref_point) return fail(BO_ERR_INVALID_ARGUMENT, W + ": ref_point is NULL");
  if (!all_finite(ref_point, M.m)) return fail(BO_ERR_NONFINITE_INPUT, W + ": ref_point not finite");
  if (M_ > (int64_t)1 << 40) return fail(BO_ERR_CAPACITY, W + ": M too large");
  if (feas_lower) {
    for (int k = 0; k < M.m; ++k)
      if (std::isnan(feas_lower[k]))
        return fail(BO_ERR_NONFINITE_INPUT, W + ": feasibility threshold is NaN");
  }
  return BO_OK;
}

// Device pointers of a scoring call (the model's device must be current).
bo_status score_check_pointers(const Model& M, const float* cand, int64_t M_, int q,
                               const float* base_samples, int S, const float* ehvi,
                               const float* mu, const float* sigma) {
  const int64_t npts = M_ * q;
  bo_status s;
  if ((s = check_dev(cand, sizeof(float) * npts * M.d, "cand")) != BO_OK) return s;
  if ((s = check_dev(base_samples, sizeof(float) * (size_t)S * q * M.m, "base_samples")) != BO_OK) return s;
  if ((s = check_dev(ehvi, sizeof(float) * M_, "ehvi")) != BO_OK) return s;
  if (mu && (s = check_dev(mu, sizeof(float) * npts * M.m, "mu")) != BO_OK) return s;
  if (sigma && (s = check_dev(sigma, sizeof(float) * npts * M.m, "sigma")) != BO_OK) return s;
  if (posterior_lds_bytes(M.nb, q) > kLdsLimit)
    return fail(BO_ERR_CAPACITY, "bo_score: posterior tile exceeds LDS");
  return BO_OK;
}

// The disjoint boxes of the region the model's front (points strictly above
// ref) does not dominate, staged as [nbox][2m] (lower corners, then widths;
// +inf widths stay +inf), with the capacity checks of a scoring call.
bo_status host_score_boxes(const Model& M, const float* ref_point, int S, int q,
                           std::vector<float>& staged, int* nbox_out) {
  const int m = M.m;
  std::vector<float> F;
  for (int32_t i : M.nd) {
    const float* y = &M.Yh[(size_t)i * m];
    bool above = true;
    for (int k = 0; k < m; ++k) above = above && (y[k] > ref_point[k]);
    if (above) F.insert(F.end(), y, y + m);
  }
  std::vector<float> lo, hi;
  host_boxes(F.data(), static_cast<int>(F.size() / m), m, ref_point, lo, hi);
  const int nbox = static_cast<int>(lo.size() / m);
  if (nbox > BO_MAX_BOXES) return fail(BO_ERR_CAPACITY, "bo_score: too many boxes");
  if (ehvi_lds_bytes(S, q, m, nbox) > kLdsLimit)
    return fail(BO_ERR_CAPACITY, "bo_score: samples and boxes exceed LDS");
  staged.resize((size_t)nbox * 2 * m);
  for (int c = 0; c < nbox; ++c)
    for (int k = 0; k < m; ++k) {
      const float l = lo[(size_t)c * m + k], h = hi[(size_t)c * m + k];
      staged[(size_t)c * 2 * m + k] = l;
      staged[(size_t)c * 2 * m + m + k] = h - l;     // inf stays inf
    }
  *nbox_out = nbox;
  return BO_OK;
}

// Floats of scoring workspace: mu and sigma [M q][m] unless the caller takes
// them, and the batch factors [M][m][q(q+1)/2] for q > 1.
size_t score_workspace_floats(const Model& M, int64_t M_, int q, bool have_mu, bool have_sigma) {
  const int64_t npts = M_ * q;
  const int T = q * (q + 1) / 2;
  return (have_mu ? 0 : (size_t)npts * M.m) + (have_sigma ? 0 : (size_t)npts * M.m) +
         (q > 1 ? (size_t)M_ * M.m * T : 0);
}

// The kernels of one scoring call on stream st: the posterior of every
// objective (into mu_buf, sd_buf and, for q > 1, chol_buf [m][M_][T]), then
// the EHVI over `boxes` (device, [nbox][2m]). mu_buf and sd_buf are the
// caller's [npts][m] arrays when mu_user / sd_user, else planar [m][npts]
// workspace, so that each objective's launch writes whole cache lines.
// rec (optional) gets profile events.
bo_status score_launches(const Model& M, const float* cand, int64_t M_, int q,
                         const float* feas_lower, const float* base_samples, int S,
                         const float* boxes, int nbox, float* ehvi, float* mu_buf, bool mu_user,
                         float* sd_buf, bool sd_user, float* chol_buf, hipStream_t st,
                         Profile::Rec* rec) {
  const int m = M.m;
  const int64_t npts = M_ * q;
  const int T = q * (q + 1) / 2;
  const int64_t mu_ps = mu_user ? m : 1, mu_ks = mu_user ? 1 : npts;
  const int64_t sd_ps = sd_user ? m : 1, sd_ks = sd_user ? 1 : npts;
  bo_status s;
  if (rec) {
    rec->launches = m;
    hipError_t e = hipEventRecord(rec->e[0], st);
    if (e != hipSuccess) return hip_fail(e, "bo_score: profile event");
  }
  for (int k = 0; k < m; ++k) {
    PosteriorArgs pa = posterior_args(M, k, M.Lp, cand, npts, q);
    pa.mu = mu_buf + k * mu_ks; pa.mu_ps = mu_ps;
    pa.sd = sd_buf + k * sd_ks; pa.sd_ps = sd_ps;
    pa.chol = chol_buf ? chol_buf + (size_t)k * M_ * T : nullptr;
    const hipError_t e = M.f64 ? launch_posterior_f64(pa, st) : launch_posterior(pa, st);
    if ((s = after_launch(e, st, "posterior")) != BO_OK) return s;
  }
  if (rec) {
    hipError_t e = hipEventRecord(rec->e[1], st);
    if (e != hipSuccess) return hip_fail(e, "bo_score: profile event");
  }
  EhviArgs ea;
  ea.mu = mu_buf; ea.sd = sd_buf; ea.chol = chol_buf;
  ea.mu_ps = mu_ps; ea.mu_ks = mu_ks; ea.sd_ps = sd_ps; ea.sd_ks = sd_ks;
  ea.Z = base_samples; ea.boxes = boxes;
  ea.nbat = M_; ea.q = q; ea.m = m; ea.S = S; ea.nbox = nbox;
  ea.constrained = feas_lower != nullptr;
  for (int k = 0; k < 3; ++k)
    ea.lower[k] = (feas_lower && k < m) ? feas_lower[k] : -INFINITY;
  ea.ehvi = ehvi;
  if ((s = after_launch(launch_ehvi(ea, st), st, "ehvi")) != BO_OK) return s;
  if (rec) {
    hipError_t e = hipEventRecord(rec->e[2], st);
    if (e != hipSuccess) return hip_fail(e, "bo_score: profile event");
  }
  return BO_OK;
}

struct CompositeSpec {
  int dr;
  const float* s_dep;
  const float* s_int;
  const float* pref;   // [m][d - dr]
};

bo_status fit_impl(const char* who, const float* X, const float* Y, int64_t n, int32_t d,
                   int32_t m, const float* lengthscale, const float* outputscale,
                   const float* noise, const CompositeSpec* comp, void* stream,
                   bo_model* out, bool f64 = false) {
  const std::string W(who);
  if (!out) return fail(BO_ERR_INVALID_ARGUMENT, W + ": out is NULL");
  if (!lengthscale || !outputscale || !noise)
    return fail(BO_ERR_INVALID_ARGUMENT, W + ": NULL hyperparameter pointer");
  if (n < 1 || d < 1 || (m != 2 && m != 3))
    return fail(BO_ERR_INVALID_ARGUMENT, W + ": need n >= 1, d >= 1, m in {2,3}");
  if (n > BO_MAX_N || d > BO_MAX_D)
    return fail(BO_ERR_CAPACITY, W + ": n or d beyond compiled limits");
  if (!all_finite(lengthscale, (size_t)m * d) || !all_finite(outputscale, m) ||
      !all_finite(noise, m))
    return fail(BO_ERR_NONFINITE_INPUT, W + ": non-finite hyperparameter");
  for (int i = 0; i < m * d; ++i)
    if (!(lengthscale[i] > 0.f)) return fail(BO_ERR_INVALID_ARGUMENT, W + ": lengthscale <= 0");
  for (int k = 0; k < m; ++k) {
    if (!(outputscale[k] > 0.f)) return fail(BO_ERR_INVALID_ARGUMENT, W + ": outputscale <= 0");
    if (!(noise[k] >= 0.f)) return fail(BO_ERR_INVALID_ARGUMENT, W + ": noise < 0");
    if (!(outputscale[k] >= kScaleMin && outputscale[k] <= kScaleMax) || !(noise[k] <= kScaleMax))
      return fail(BO_ERR_INVALID_ARGUMENT,
                  W + ": outputscale outside [2^-64, 2^64] or noise above 2^64");
  }
  int dr = 0, dr4 = 0, dx = (d + 3) / 4 * 4;
  if (comp) {
    dr = comp->dr;
    if (dr < 1 || dr >= d)
      return fail(BO_ERR_INVALID_ARGUMENT, W + ": need 1 <= d_route < d");
    if (!comp->s_dep || !comp->s_int || !comp->pref)
      return fail(BO_ERR_INVALID_ARGUMENT, W + ": NULL hyperparameter pointer");
    if (!all_finite(comp->s_dep, m) || !all_finite(comp->s_int, m) ||
        !all_finite(comp->pref, (size_t)m * (d - dr)))
      return fail(BO_ERR_NONFINITE_INPUT, W + ": non-finite hyperparameter");
    for (int k = 0; k < m; ++k) {
      if (!(comp->s_dep[k] >= 0.f) || !(comp->s_int[k] >= 0.f))
        return fail(BO_ERR_INVALID_ARGUMENT, W + ": scale_dep / scale_int < 0");
      if (!(comp->s_dep[k] <= kScaleMax) || !(comp->s_int[k] <= kScaleMax))
        return fail(BO_ERR_INVALID_ARGUMENT, W + ": scale_dep / scale_int above 2^64");
    }
    dr4 = (dr + 3) / 4;
    dx = 4 * dr4 + (d - dr + 3) / 4 * 4;
    if (dx > BO_MAX_D)
      return fail(BO_ERR_CAPACITY, W + ": padded routing + deployment groups exceed BO_MAX_D");
  }
  bo_status s;
  if ((s = check_dev(X, sizeof(float) * n * d, "X")) != BO_OK) return s;
  if ((s = check_dev(Y, sizeof(float) * n * m, "Y")) != BO_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);

  bo_model_s* h = new (std::nothrow) bo_model_s();
  if (!h) return fail(BO_ERR_OUT_OF_MEMORY, W + ": host allocation");
  Model* M = &h->m;
  (void)hipGetDevice(&M->device);
  M->n = n; M->d = d; M->m = m;
  M->n_pad = static_cast<int>((n + kBlk - 1) / kBlk) * kBlk;
  M->nb = M->n_pad / kBlk;
  M->dx = dx;
  M->dr = dr; M->dr4 = dr4;
  M->f64 = f64;
  M->ls.assign(lengthscale, lengthscale + (size_t)m * d);
  M->os.assign(outputscale, outputscale + m);
  M->noise.assign(noise, noise + m);
  if (comp) {
    M->s_dep.assign(comp->s_dep, comp->s_dep + m);
    M->s_int.assign(comp->s_int, comp->s_int + m);
    M->prefh.assign(comp->pref, comp->pref + (size_t)m * (d - comp->dr));
  }

  auto bail = [&](bo_status st_) {
    release_buffers(M);
    delete h;
    return st_;
  };

  const int nf = static_cast<int>((n + kFitBlk - 1) / kFitBlk) * kFitBlk;
  const int dc = d - dr;
  M->lp_per_obj = packed_factor_floats(M->nb);
  // fp64 hyperparameters: [1/ls m*d][os m][noise m] (+ [s_dep m][s_int m][pref m*dc])
  const size_t nhyp = (size_t)m * d + 2 * m + (comp ? 2 * m + (size_t)m * dc : 0);
  // every model buffer in one allocation
  ArenaLayout lay;
  const size_t o_xs = lay.add(sizeof(float) * m * M->n_pad * M->dx);
  const size_t o_il = lay.add(sizeof(float) * m * M->dx);
  const size_t o_al = lay.add(sizeof(float) * m * M->n_pad);
  const size_t o_lp = lay.add(sizeof(float) * m * M->lp_per_obj);
  const size_t o_xd = lay.add(sizeof(float) * n * d);
  const size_t o_xf = lay.add(sizeof(uint16_t) * m * M->nb * dist_frags(M->dx) * 512);
  const size_t o_x2 = lay.add(sizeof(float) * m * 2 * M->n_pad);
  const size_t o_ct = lay.add(sizeof(float) * m * M->dx);
  size_t o_l64 = 0, o_a64 = 0, o_i64 = 0, o_wt = 0, o_pf = 0;
  if (f64) {
    o_l64 = lay.add(sizeof(double) * m * posterior_f64_blocks(M->nb) * 512);
    o_a64 = lay.add(sizeof(double) * m * nf);
    o_i64 = lay.add(sizeof(double) * m * d);
  }
  if (comp) {
    o_wt = lay.add(sizeof(float) * m * M->n_pad);
    o_pf = lay.add(sizeof(float) * m * dc);
  }
  {
    // the device's spare allocation when it is large enough, else a new one
    DeviceState* DSa = device_state(M->device);
    if (!DSa) return bail(fail(BO_ERR_DEVICE, W + ": device index out of range"));
    std::lock_guard<std::mutex> lk(DSa->mu);
    if (DSa->spare && DSa->spare_bytes >= lay.total) {
      M->arena = DSa->spare;
      M->arena_bytes = DSa->spare_bytes;
      DSa->spare = nullptr;
      DSa->spare_bytes = 0;
    }
  }
  if (!M->arena) {
    if ((s = palloc(&M->arena, lay.total, st, "model buffers")) != BO_OK) return bail(s);
    M->arena_bytes = lay.total;
  }
  M->pending = true;   // until the fit's work is known to be complete
  {
    unsigned char* b = M->arena;
    M->Xs = reinterpret_cast<float*>(b + o_xs);
    M->invls = reinterpret_cast<float*>(b + o_il);
    M->alpha = reinterpret_cast<float*>(b + o_al);
    M->Lp = reinterpret_cast<float*>(b + o_lp);
    M->Xd = reinterpret_cast<float*>(b + o_xd);
    M->xf = reinterpret_cast<uint16_t*>(b + o_xf);
    M->x2 = reinterpret_cast<float*>(b + o_x2);
    M->ctr = reinterpret_cast<float*>(b + o_ct);
    if (f64) {
      M->Lp64 = reinterpret_cast<double*>(b + o_l64);
      M->alpha64 = reinterpret_cast<double*>(b + o_a64);
      M->ils64 = reinterpret_cast<double*>(b + o_i64);
    }
    if (comp) {
      M->wts = reinterpret_cast<float*>(b + o_wt);
      M->pref = reinterpret_cast<float*>(b + o_pf);
    }
  }
  M->n_fit = nf;

  std::vector<double> hyp(nhyp);
  for (int i = 0; i < m * d; ++i) hyp[i] = 1.0 / static_cast<double>(lengthscale[i]);
  for (int k = 0; k < m; ++k) {
    hyp[(size_t)m * d + k] = outputscale[k];
    hyp[(size_t)m * d + m + k] = noise[k];
    if (comp) {
      hyp[(size_t)m * d + 2 * m + k] = comp->s_dep[k];
      hyp[(size_t)m * d + 3 * m + k] = comp->s_int[k];
    }
  }
  if (comp)
    for (size_t i = 0; i < (size_t)m * dc; ++i) hyp[(size_t)m * d + 4 * m + i] = comp->pref[i];

  // pinned staging mirrors the device scratch from the hyperparameters on:
  // [hyperparameters, zero padding to hyp_cap][flag, statistics, maxima
  // (zeros going up; flag and statistics come back here)][Y]
  DeviceState* DS = device_state(M->device);
  if (!DS) return bail(fail(BO_ERR_DEVICE, W + ": device index out of range"));
  std::lock_guard<std::mutex> stage_lock(DS->fit_mu);
  FitScratch fs;
  fs.st = st;
  if ((s = fit_work(DS, (size_t)m * nf * nf, nhyp, (size_t)m * nf, &fs)) != BO_OK) return bail(s);
  const size_t off_flag = sizeof(double) * fs.hyp_cap;
  const size_t off_stats = off_flag + 16;
  const size_t up_bytes = off_flag + kFitSmall;
  const size_t off_y = (up_bytes + 15) / 16 * 16;
  const size_t need = off_y + sizeof(float) * n * m;
  hipError_t e = hipSuccess;
  if (need > DS->fit_stage_bytes) {
    if (DS->fit_stage) (void)hipHostFree(DS->fit_stage);
    DS->fit_stage = nullptr;
    DS->fit_stage_bytes = 0;
    const size_t cap = std::max<size_t>(need, size_t(1) << 16);
    e = hipHostMalloc(reinterpret_cast<void**>(&DS->fit_stage), cap, hipHostMallocDefault);
    if (e != hipSuccess) return bail(hip_fail(e, "bo_fit: pinned staging"));
    DS->fit_stage_bytes = cap;
  }
  unsigned char* stage = DS->fit_stage;
  std::memcpy(stage, hyp.data(), sizeof(double) * hyp.size());
  std::memset(stage + sizeof(double) * hyp.size(), 0, up_bytes - sizeof(double) * hyp.size());
  // the fp32 inverse lengthscales and preference slopes, and the copy of X,
  // are written on the device from these (k_scale_x); the flag, statistics
  // and maxima start at zero
  e = hipMemcpyAsync(fs.hyp, stage, up_bytes, hipMemcpyHostToDevice, st);
  // Y comes back first, so that its finiteness check and the front run on
  // the host while the device factors
  if (e == hipSuccess && !DS->fit_evt) e = hipEventCreateWithFlags(&DS->fit_evt, hipEventDisableTiming);
  if (e == hipSuccess)
    e = hipMemcpyAsync(stage + off_y, Y, sizeof(float) * n * m, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipEventRecord(DS->fit_evt, st);
  if (e != hipSuccess) return bail(hip_fail(e, "bo_fit: upload"));

  GramParams gp;
  gp.dr = dr;
  gp.ils = fs.hyp;
  gp.os = fs.hyp + (size_t)m * d;
  gp.noise = gp.os + m;
  if (comp) {
    gp.s_dep = gp.noise + m;
    gp.s_int = gp.s_dep + m;
    gp.pref = gp.s_int + m;
  }
  // The Gram matrix past its first 64 columns, the scaled X, its distance
  // fragments and (composite) the preference weights depend only on X and
  // the hyperparameters: they run on the side stream beside the first
  // diagonal block's factor and panel (the first trailing update waits for
  // the Gram columns), and the side stream joins once the factorisation is
  // done; the fp16 pack and alpha then follow on this stream (alpha on the
  // side stream, beside the pack, took longer: its wait for the factor cost
  // more than the pack). (An event's later record does not change a wait
  // already enqueued on it.)
  if ((s = side_stream(DS)) != BO_OK) return bail(s);
  hipStream_t side = DS->side;
  e = hipEventRecord(DS->side_evt[0], st);
  if (e == hipSuccess) e = hipStreamWaitEvent(side, DS->side_evt[0], 0);
  if (e != hipSuccess) return bail(hip_fail(e, "bo_fit: side stream"));
  // enqueued in the order the device should start them: the critical chain
  // first (the first block column of the Gram matrix, then the factor,
  // which waits for the rest of the Gram matrix before its first update)
  if ((s = after_launch(launch_gram(X, n, d, m, nf, gp, fs.A, st, fs.stats, 0, kFitBlk), st, "gram")) != BO_OK) return bail(s);
  if ((s = after_launch(launch_gram(X, n, d, m, nf, gp, fs.A, side, fs.stats, kFitBlk, nf), side, "gram")) != BO_OK) return bail(s);
  e = hipEventRecord(DS->side_evt[2], side);
  if (e != hipSuccess) return bail(hip_fail(e, "bo_fit: side stream"));
  if ((s = after_launch(launch_cholesky(fs.A, fs.W, nf, m, fs.flag, st, DS->side_evt[2]), st, "cholesky")) != BO_OK) return bail(s);
  if ((s = after_launch(launch_scale_x(X, n, d, m, M->nb, M->dx, dr, dr4, gp.ils, M->invls,
                                       comp ? gp.pref : nullptr, M->pref, M->Xd, M->ils64,
                                       M->Xs, side), side, "scale X")) != BO_OK) return bail(s);
  if ((s = after_launch(launch_pack_x(M->Xs, n, m, M->nb, M->dx, dr4, M->ctr, M->xf, M->x2, side), side, "pack X")) != BO_OK) return bail(s);
  if (comp && (s = after_launch(launch_weights(X, n, d, m, M->n_pad, gp, M->wts, side), side, "weights")) != BO_OK) return bail(s);
  // alpha (and the fp64 fragments) and the fp16 pack on this stream; the side
  // stream's work joins first
  e = hipEventRecord(DS->side_evt[1], side);
  if (e == hipSuccess) e = hipStreamWaitEvent(st, DS->side_evt[1], 0);
  if (e != hipSuccess) return bail(hip_fail(e, "bo_fit: side stream"));
  if ((s = after_launch(launch_pack_factor(fs.W, n, m, nf, M->nb, M->Lp, fs.stats + m, fs.flag, st, fs.bmax), st, "pack")) != BO_OK) return bail(s);
  if ((s = after_launch(launch_alpha(fs.W, Y, n, m, nf, M->n_pad, fs.tmp, M->alpha, st, M->alpha64), st, "alpha")) != BO_OK) return bail(s);
  if (f64 && (s = after_launch(launch_pack_f64(fs.W, n, m, nf, M->nb, M->Lp64, st), st, "pack fp64")) != BO_OK) return bail(s);

  // the flag and statistics follow the work; Y (copied back first) is
  // checked and its front formed meanwhile, then one synchronisation
  e = hipMemcpyAsync(stage + off_flag, fs.flag, 64, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipEventSynchronize(DS->fit_evt);
  if (e != hipSuccess) return bail(hip_fail(e, "bo_fit: read-back"));
  const float* yst = reinterpret_cast<const float*>(stage + off_y);
  M->Yh.assign(yst, yst + (size_t)n * m);
  if (!all_finite(M->Yh.data(), M->Yh.size()))
    return bail(fail(BO_ERR_NONFINITE_INPUT, W + ": Y not finite"));
  host_front<float>(M->Yh.data(), n, m, nullptr, M->nd);
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return bail(hip_fail(e, "bo_fit: sync"));
  M->pending = false;   // every kernel of the fit has finished
  int flag = 0;
  std::memcpy(&flag, stage + off_flag, sizeof(int));
  if (flag)
    return bail(fail(BO_ERR_NOT_POSITIVE_DEFINITE,
                     W + ": non-positive Cholesky pivot or non-finite inverse factor"));
  {
    unsigned long long st_bits[6];
    std::memcpy(st_bits, stage + off_stats, sizeof(unsigned long long) * 2 * m);
    M->kbound.resize(m);
    M->cond_est.resize(m);
    for (int k = 0; k < m; ++k) {
      const double kd = bits_to_double(st_bits[k]), wm = bits_to_double(st_bits[m + k]);
      M->kbound[k] = static_cast<float>(kd);
      M->cond_est[k] = kd * wm * wm;
      if (!(M->cond_est[k] < (f64 ? kCondLimitF64 : kCondLimit))) {
        char msg[200];
        std::snprintf(msg, sizeof msg,
                      ": objective %d: max K_ii * max |L^-1|^2 = %.3g reaches %s (a lower "
                      "bound on cond(K)); the %s scoring cannot resolve this model",
                      k, M->cond_est[k], f64 ? "2^50" : "2^24", f64 ? "fp64" : "fp32-class");
        return bail(fail(BO_ERR_ILL_CONDITIONED, W + msg));
      }
    }
  }

  M->last_stream = st;
  *out = h;
  return BO_OK;
}

// Log marginal likelihood and gradient: the fit's Gram, factor and alpha in
// fp64, then the likelihood kernels; no model is kept.
bo_status mll_impl(const float* X, const float* Y, int64_t n, int32_t d, int32_t m,
                   const float* lengthscale, const float* outputscale, const float* noise,
                   void* stream, double* value, double* grad) {
  if (!value || !grad) return fail(BO_ERR_INVALID_ARGUMENT, "bo_mll: NULL output");
  if (!lengthscale || !outputscale || !noise)
    return fail(BO_ERR_INVALID_ARGUMENT, "bo_mll: NULL hyperparameter pointer");
  if (n < 1 || d < 1 || (m != 2 && m != 3))
    return fail(BO_ERR_INVALID_ARGUMENT, "bo_mll: need n >= 1, d >= 1, m in {2,3}");
  if (n > BO_MAX_N || d > BO_MAX_D)
    return fail(BO_ERR_CAPACITY, "bo_mll: n or d beyond compiled limits");
  if (!all_finite(lengthscale, (size_t)m * d) || !all_finite(outputscale, m) ||
      !all_finite(noise, m))
    return fail(BO_ERR_NONFINITE_INPUT, "bo_mll: non-finite hyperparameter");
  for (int i = 0; i < m * d; ++i)
    if (!(lengthscale[i] > 0.f)) return fail(BO_ERR_INVALID_ARGUMENT, "bo_mll: lengthscale <= 0");
  for (int k = 0; k < m; ++k) {
    if (!(outputscale[k] > 0.f)) return fail(BO_ERR_INVALID_ARGUMENT, "bo_mll: outputscale <= 0");
    if (!(noise[k] >= 0.f)) return fail(BO_ERR_INVALID_ARGUMENT, "bo_mll: noise < 0");
  }
  bo_status s;
  if ((s = check_dev(X, sizeof(float) * n * d, "X")) != BO_OK) return s;
  if ((s = check_dev(Y, sizeof(float) * n * m, "Y")) != BO_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  int dev = 0;
  (void)hipGetDevice(&dev);

  const int nf = static_cast<int>((n + kFitBlk - 1) / kFitBlk) * kFitBlk;
  const int n_pad = static_cast<int>((n + kBlk - 1) / kBlk) * kBlk;
  const int64_t tiles = mll_tiles(nf);
  struct Extra {
    hipStream_t st = nullptr;
    float* alpha = nullptr;
    double* alpha64 = nullptr;
    double* partials = nullptr;
    double* out = nullptr;
    ~Extra() { pfree(alpha, st); pfree(alpha64, st); pfree(partials, st); pfree(out, st); }
  } ex;
  ex.st = st;
  const size_t nhyp = (size_t)m * d + 2 * m;
  if ((s = palloc(&ex.alpha, (size_t)m * n_pad, st, "alpha")) != BO_OK) return s;
  if ((s = palloc(&ex.alpha64, (size_t)m * nf, st, "alpha (fp64)")) != BO_OK) return s;
  if ((s = palloc(&ex.partials, (size_t)m * tiles * (d + 2), st, "gradient partials")) != BO_OK) return s;
  if ((s = palloc(&ex.out, (size_t)m * (d + 3), st, "likelihood")) != BO_OK) return s;

  std::vector<double> hyp(nhyp);
  for (int i = 0; i < m * d; ++i) hyp[i] = 1.0 / static_cast<double>(lengthscale[i]);
  for (int k = 0; k < m; ++k) {
    hyp[(size_t)m * d + k] = outputscale[k];
    hyp[(size_t)m * d + m + k] = noise[k];
  }
  // pinned staging: [hyperparameters][flag][value, gradient]
  DeviceState* DS = device_state(dev);
  if (!DS) return fail(BO_ERR_DEVICE, "bo_mll: device index out of range");
  std::lock_guard<std::mutex> stage_lock(DS->fit_mu);
  FitScratch fs;
  fs.st = st;
  if ((s = fit_work(DS, (size_t)m * nf * nf, nhyp, (size_t)m * nf, &fs)) != BO_OK) return s;
  const size_t off_flag = (sizeof(double) * nhyp + 15) / 16 * 16;
  const size_t off_out = off_flag + 16;
  const size_t need = off_out + sizeof(double) * m * (d + 3);
  hipError_t e = hipSuccess;
  if (need > DS->fit_stage_bytes) {
    if (DS->fit_stage) (void)hipHostFree(DS->fit_stage);
    DS->fit_stage = nullptr;
    DS->fit_stage_bytes = 0;
    const size_t cap = std::max<size_t>(need, size_t(1) << 16);
    e = hipHostMalloc(reinterpret_cast<void**>(&DS->fit_stage), cap, hipHostMallocDefault);
    if (e != hipSuccess) return hip_fail(e, "bo_mll: pinned staging");
    DS->fit_stage_bytes = cap;
  }
  unsigned char* stage = DS->fit_stage;
  std::memcpy(stage, hyp.data(), sizeof(double) * nhyp);
  auto sync_fail = [&](bo_status st_) {
    (void)hipStreamSynchronize(st);   // copies from the staging buffer may be pending
    return st_;
  };
  e = hipMemcpyAsync(fs.hyp, stage, sizeof(double) * nhyp, hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipMemsetAsync(fs.flag, 0, sizeof(int), st);
  if (e != hipSuccess) return sync_fail(hip_fail(e, "bo_mll: upload"));

  GramParams gp;
  gp.ils = fs.hyp;
  gp.os = fs.hyp + (size_t)m * d;
  gp.noise = gp.os + m;
  if ((s = after_launch(launch_gram(X, n, d, m, nf, gp, fs.A, st), st, "gram")) != BO_OK) return sync_fail(s);
  if ((s = after_launch(launch_cholesky(fs.A, fs.W, nf, m, fs.flag, st), st, "cholesky")) != BO_OK) return sync_fail(s);
  if ((s = after_launch(launch_alpha(fs.W, Y, n, m, nf, n_pad, fs.tmp, ex.alpha, st, ex.alpha64), st, "alpha")) != BO_OK) return sync_fail(s);
  if ((s = after_launch(launch_mll(X, n, d, m, nf, gp, fs.A, fs.W, fs.tmp, ex.alpha64, ex.partials, ex.out, st), st, "likelihood")) != BO_OK) return sync_fail(s);
  e = hipMemcpyAsync(stage + off_flag, fs.flag, sizeof(int), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(stage + off_out, ex.out, sizeof(double) * m * (d + 3), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "bo_mll: sync");
  int flag = 0;
  std::memcpy(&flag, stage + off_flag, sizeof(int));
  if (flag) return fail(BO_ERR_NOT_POSITIVE_DEFINITE, "bo_mll: non-positive Cholesky pivot");
  const double* o = reinterpret_cast<const double*>(stage + off_out);
  for (int k = 0; k < m; ++k) {
    value[k] = o[k * (d + 3)];
    for (int j = 0; j < d + 2; ++j) grad[(size_t)k * (d + 2) + j] = o[k * (d + 3) + 1 + j];
  }
  return BO_OK;
}

}  // namespace

extern "C" {

bo_status bo_mll(const float* X, const float* Y, int64_t n, int32_t d, int32_t m,
                 const float* lengthscale, const float* outputscale, const float* noise,
                 void* stream, double* value, double* grad) {
  return mll_impl(X, Y, n, d, m, lengthscale, outputscale, noise, stream, value, grad);
}

bo_status bo_fit(const float* X, const float* Y, int64_t n, int32_t d, int32_t m,
                 const float* lengthscale, const float* outputscale, const float* noise,
                 void* stream, bo_model* out) {
  return fit_impl("bo_fit", X, Y, n, d, m, lengthscale, outputscale, noise, nullptr, stream,
                  out);
}

bo_status bo_fit_composite(const float* X, const float* Y, int64_t n, int32_t d, int32_t m,
                           int32_t d_route, const float* lengthscale,
                           const float* scale_route, const float* scale_dep,
                           const float* scale_int, const float* pref, const float* noise,
                           void* stream, bo_model* out) {
  const CompositeSpec c{d_route, scale_dep, scale_int, pref};
  return fit_impl("bo_fit_composite", X, Y, n, d, m, lengthscale, scale_route, noise, &c,
                  stream, out);
}

bo_status bo_fit_f64(const float* X, const float* Y, int64_t n, int32_t d, int32_t m,
                     const float* lengthscale, const float* outputscale, const float* noise,
                     void* stream, bo_model* out) {
  return fit_impl("bo_fit_f64", X, Y, n, d, m, lengthscale, outputscale, noise, nullptr, stream,
                  out, true);
}

bo_status bo_fit_composite_f64(const float* X, const float* Y, int64_t n, int32_t d, int32_t m,
                               int32_t d_route, const float* lengthscale,
                               const float* scale_route, const float* scale_dep,
                               const float* scale_int, const float* pref, const float* noise,
                               void* stream, bo_model* out) {
  const CompositeSpec c{d_route, scale_dep, scale_int, pref};
  return fit_impl("bo_fit_composite_f64", X, Y, n, d, m, lengthscale, scale_route, noise, &c,
                  stream, out, true);
}

void bo_free(bo_model model) {
  if (!model) return;
  DeviceGuard g(model->m.device);
  release_buffers(&model->m);
  if (model->m.last_evt) (void)hipEventDestroy(model->m.last_evt);
  delete model;
}

bo_status bo_score(bo_model model, const float* cand, int64_t M_, int32_t q,
                   const float* ref_point, const float* base_samples, int32_t S,
                   float* ehvi, float* mu, float* sigma, void* stream) {
  return bo_score_constrained(model, cand, M_, q, ref_point, nullptr, base_samples, S, ehvi,
                              mu, sigma, stream);
}

bo_status bo_score_constrained(bo_model model, const float* cand, int64_t M_, int32_t q,
                               const float* ref_point, const float* feas_lower,
                               const float* base_samples, int32_t S, float* ehvi, float* mu,
                               float* sigma, void* stream) {
  bo_status s;
  if ((s = score_validate("bo_score", model, cand, M_, q, ref_point, feas_lower, base_samples, S,
                          ehvi, mu, sigma)) != BO_OK)
    return s;
  Model& M = model->m;
  if (M_ == 0) return BO_OK;
  DeviceGuard g(M.device);
  if (!g.ok) return fail(BO_ERR_DEVICE, "bo_score: cannot select the model's device");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int m = M.m;
  const int64_t npts = M_ * q;
  if ((s = score_check_pointers(M, cand, M_, q, base_samples, S, ehvi, mu, sigma)) != BO_OK) return s;
  if ((s = order_after_previous(M, st, "bo_score: stream ordering")) != BO_OK) return s;

  // ---- boxes (host, cached per reference point) ------------------------
  const bool same_ref = M.nbox >= 0 && M.box_ref.size() == (size_t)m &&
                        std::memcmp(M.box_ref.data(), ref_point, sizeof(float) * m) == 0;
  if (!same_ref) {
    std::vector<float> staged;
    int nbox = 0;
    if ((s = host_score_boxes(M, ref_point, S, q, staged, &nbox)) != BO_OK) return s;
    if (nbox > M.box_cap) {
      if (M.d_boxes) {
        hipError_t e = hipDeviceSynchronize();   // earlier launches may read it
        if (e != hipSuccess) return hip_fail(e, "bo_score: sync before box growth");
        pfree(M.d_boxes, st);
      }
      M.box_cap = 0;
      const int cap = std::max(64, nbox);
      if ((s = palloc(&M.d_boxes, (size_t)cap * 2 * m, st, "boxes")) != BO_OK) return s;
      M.box_cap = cap;
    }
    {
      // stage in the device's pinned buffer; the previous upload from it must
      // have completed before it is rewritten
      DeviceState* DS = device_state(M.device);
      std::lock_guard<std::mutex> lk(DS->mu);
      hipError_t e = hipSuccess;
      if (!DS->stage_evt) e = hipEventCreateWithFlags(&DS->stage_evt, hipEventDisableTiming);
      else e = hipEventSynchronize(DS->stage_evt);
      if (e != hipSuccess) return hip_fail(e, "bo_score: staging event");
      const size_t need_f = staged.size();
      if (need_f > DS->stage_floats) {
        if (DS->stage) (void)hipHostFree(DS->stage);
        DS->stage = nullptr;
        DS->stage_floats = 0;
        const size_t cap = std::max<size_t>(need_f, (size_t)BO_MAX_BOXES * 6);
        e = hipHostMalloc(reinterpret_cast<void**>(&DS->stage), sizeof(float) * cap, hipHostMallocDefault);
        if (e != hipSuccess) return hip_fail(e, "bo_score: pinned staging");
        DS->stage_floats = cap;
      }
      std::memcpy(DS->stage, staged.data(), sizeof(float) * need_f);
      e = hipMemcpyAsync(M.d_boxes, DS->stage, sizeof(float) * need_f, hipMemcpyHostToDevice, st);
      if (e == hipSuccess) e = hipEventRecord(DS->stage_evt, st);
      if (e != hipSuccess) return hip_fail(e, "bo_score: box upload");
    }
    M.nbox = nbox;
    M.box_ref.assign(ref_point, ref_point + m);
  } else if (ehvi_lds_bytes(S, q, m, M.nbox) > kLdsLimit) {
    return fail(BO_ERR_CAPACITY, "bo_score: samples and boxes exceed LDS");
  }

  // ---- workspace ----------------------------------------------------------
  const size_t need = score_workspace_floats(M, M_, q, mu != nullptr, sigma != nullptr);
  if (need > M.ws_floats) {
    if (M.ws) {
      hipError_t e = hipDeviceSynchronize();      // earlier launches may use it
      if (e != hipSuccess) return hip_fail(e, "bo_score: sync before workspace growth");
      pfree(M.ws, st);
    }
    M.ws_floats = 0;
    if ((s = palloc(&M.ws, need, st, "score workspace")) != BO_OK) return s;
    M.ws_floats = need;
  }
  float* w = M.ws;
  float* mu_buf = mu ? mu : w;
  if (!mu) w += (size_t)npts * m;
  float* sd_buf = sigma ? sigma : w;
  if (!sigma) w += (size_t)npts * m;
  float* chol_buf = (q > 1) ? w : nullptr;

  // ---- launches -------------------------------------------------------------
  Profile::Rec* rec = nullptr;
  {
    Profile& P = profile();
    std::lock_guard<std::mutex> lk(P.mu);
    if (P.on && P.used < P.pool.size()) rec = &P.pool[P.used++];
  }
  if ((s = score_launches(M, cand, M_, q, feas_lower, base_samples, S, M.d_boxes, M.nbox, ehvi,
                          mu_buf, mu != nullptr, sd_buf, sigma != nullptr, chol_buf, st, rec)) != BO_OK)
    return s;
  return mark_call(M, st, "bo_score: stream ordering");
}

bo_status bo_score_noalloc(bo_model model, const float* cand, int64_t M_, int32_t q,
                           const float* ref_point, const float* base_samples, int32_t S,
                           float* ehvi, void* stream) {
  bo_status s;
  if ((s = score_validate("bo_score_noalloc", model, cand, M_, q, ref_point, nullptr,
                          base_samples, S, ehvi, nullptr, nullptr)) != BO_OK)
    return s;
  Model& M = model->m;
  if (M_ == 0) return BO_OK;
  const size_t need = score_workspace_floats(M, M_, q, false, false);
  if (need > kNoallocScratchFloats - kNoallocBoxFloats)
    return fail(BO_ERR_CAPACITY, "bo_score_noalloc: M * q * m beyond the 32 MiB scratch");
  DeviceGuard g(M.device);
  if (!g.ok) return fail(BO_ERR_DEVICE, "bo_score_noalloc: cannot select the model's device");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int m = M.m;
  const int64_t npts = M_ * q;
  if ((s = score_check_pointers(M, cand, M_, q, base_samples, S, ehvi, nullptr, nullptr)) != BO_OK)
    return s;
  float* scr = nullptr;
  if ((s = noalloc_scratch(M.device, &scr)) != BO_OK) return s;
  if ((s = order_after_previous(M, st, "bo_score_noalloc: stream ordering")) != BO_OK) return s;
  // boxes into the scratch: from pageable host memory the copy completes
  // before hipMemcpyAsync returns, after the earlier work on the stream
  std::vector<float> staged;
  int nbox = 0;
  if ((s = host_score_boxes(M, ref_point, S, q, staged, &nbox)) != BO_OK) return s;
  hipError_t e = hipMemcpyAsync(scr, staged.data(), sizeof(float) * staged.size(),
                                hipMemcpyHostToDevice, st);
  if (e != hipSuccess) return hip_fail(e, "bo_score_noalloc: box upload");
  float* mu_buf = scr + kNoallocBoxFloats;
  float* sd_buf = mu_buf + (size_t)npts * m;
  float* chol_buf = (q > 1) ? sd_buf + (size_t)npts * m : nullptr;
  return score_launches(M, cand, M_, q, nullptr, base_samples, S, scr, nbox, ehvi, mu_buf, false,
                        sd_buf, false, chol_buf, st, nullptr);
}

}  // extern "C"

namespace {

// Candidates per scoring chunk of the noisy acquisition: the conditional
// means of a chunk, m x S x chunk floats (4 GiB at m = 2, S = 512), stay in HBM
// between the matrix-core kernel and the HVI kernel.
constexpr int64_t kNehviChunk = 1048576;
constexpr int kNehviMaxS = 512;

struct NoisyScratch {
  hipStream_t st = nullptr;
  double *A = nullptr, *W = nullptr, *A0 = nullptr, *W0 = nullptr;
  double *hyp = nullptr, *tmp = nullptr, *alpha64 = nullptr, *gmax = nullptr;
  double *Zk = nullptr, *T1 = nullptr, *G = nullptr, *Fd = nullptr;
  float *Y = nullptr, *alpha = nullptr, *btmp = nullptr;
  int *flag = nullptr, *counts = nullptr, *off = nullptr;
  unsigned long long* stats = nullptr;   // [2m]: max K_XX,ii, then max |L_XX^{-1}| (double bits)
  ~NoisyScratch() {
    pfree(A, st); pfree(W, st); pfree(A0, st); pfree(W0, st); pfree(hyp, st); pfree(tmp, st);
    pfree(alpha64, st); pfree(gmax, st); pfree(Zk, st); pfree(T1, st); pfree(G, st); pfree(Fd, st);
    pfree(Y, st); pfree(alpha, st); pfree(btmp, st); pfree(flag, st); pfree(counts, st);
    pfree(off, st); pfree(stats, st);
  }
};

bo_status nehvi_prepare_impl(bo_model model, const float* ZX, int32_t S, const float* ref,
                             const float* lower, void* stream) {
  const std::string W_("bo_nehvi_prepare");
  if (!model) return fail(BO_ERR_INVALID_ARGUMENT, W_ + ": model is NULL");
  Model& M = model->m;
  const int m = M.m, d = M.d;
  if (M.f64)
    return fail(BO_ERR_INVALID_ARGUMENT, W_ + ": the noisy acquisition is fp32-class only "
                                              "(fit with bo_fit or bo_fit_composite)");
  if (m != 2 && m != 3) return fail(BO_ERR_INVALID_ARGUMENT, W_ + ": two or three objectives");
  if (S < 1) return fail(BO_ERR_INVALID_ARGUMENT, W_ + ": S < 1");
  if (S > kNehviMaxS) return fail(BO_ERR_CAPACITY, W_ + ": S beyond 512");
  if (!ref) return fail(BO_ERR_INVALID_ARGUMENT, W_ + ": ref_point is NULL");
  if (!all_finite(ref, m)) return fail(BO_ERR_NONFINITE_INPUT, W_ + ": ref_point not finite");
  if (lower)
    for (int k = 0; k < m; ++k)
      if (std::isnan(lower[k])) return fail(BO_ERR_NONFINITE_INPUT, W_ + ": feasibility threshold is NaN");
  DeviceGuard g(M.device);
  if (!g.ok) return fail(BO_ERR_DEVICE, W_ + ": cannot select the model's device");
  const int64_t n = M.n;
  bo_status s;
  if ((s = check_dev(ZX, sizeof(float) * (size_t)S * n * m, "base_samples_X")) != BO_OK) return s;
  if (m == 2 && nehvi_front_lds_bytes(n) > 64 * 1024)
    return fail(BO_ERR_CAPACITY, W_ + ": n beyond the front kernel's LDS");
  if (m == 3 && nehvi_front3_lds_bytes(n) > kLdsLimit)
    return fail(BO_ERR_CAPACITY, W_ + ": n beyond the front kernel's LDS");
  hipStream_t st = static_cast<hipStream_t>(stream);
  M.pending = true;   // its launches read the model's buffers
  const int nf = static_cast<int>((n + kFitBlk - 1) / kFitBlk) * kFitBlk;
  const int Sp = nehvi_padded_samples(S);
  const int n32 = static_cast<int>((n + 31) / 32);
  const int nrb = Sp / 16;

  // earlier scoring calls may still read the state being replaced
  release_noisy(&M);
  Model::Noisy& z = M.nz;

  NoisyScratch sc;
  sc.st = st;
  // fp64 hyperparameters: [1/ls][os][noise][zeros] (+ [s_dep][s_int][pref])
  const int dc = d - M.dr;
  const bool comp = M.dr > 0;
  const size_t nhyp = (size_t)m * d + 3 * m + (comp ? 2 * (size_t)m + (size_t)m * dc : 0);
  const size_t mat = (size_t)m * nf * nf, vec = (size_t)m * nf * Sp;
  if ((s = palloc(&sc.A, mat, st, "noisy: matrix")) != BO_OK) return s;
  if ((s = palloc(&sc.W, mat, st, "noisy: inverse")) != BO_OK) return s;
  if ((s = palloc(&sc.A0, mat, st, "noisy: noise-free matrix")) != BO_OK) return s;
  if ((s = palloc(&sc.W0, mat, st, "noisy: noise-free inverse")) != BO_OK) return s;
  if ((s = palloc(&sc.hyp, nhyp, st, "noisy: hyperparameters")) != BO_OK) return s;
  if ((s = palloc(&sc.tmp, (size_t)m * nf, st, "noisy: vector")) != BO_OK) return s;
  if ((s = palloc(&sc.alpha64, (size_t)m * nf, st, "noisy: alpha")) != BO_OK) return s;
  if ((s = palloc(&sc.gmax, (size_t)m * kAbsmaxParts, st, "noisy: maxima")) != BO_OK) return s;
  if ((s = palloc(&sc.Zk, vec, st, "noisy: base samples")) != BO_OK) return s;
  if ((s = palloc(&sc.T1, vec, st, "noisy: in-sample offsets")) != BO_OK) return s;
  if ((s = palloc(&sc.G, vec, st, "noisy: G")) != BO_OK) return s;
  if ((s = palloc(&sc.Y, (size_t)n * m, st, "noisy: Y")) != BO_OK) return s;
  if ((s = palloc(&sc.alpha, (size_t)m * M.n_pad, st, "noisy: alpha (fp32)")) != BO_OK) return s;
  if ((s = palloc(&sc.flag, 8, st, "noisy: flags")) != BO_OK) return s;
  if ((s = palloc(&sc.stats, 2 * (size_t)m, st, "noisy: statistics")) != BO_OK) return s;
  if ((s = palloc(&sc.counts, 2 * (size_t)S, st, "noisy: counts")) != BO_OK) return s;
  if ((s = palloc(&sc.off, (size_t)S + 1, st, "noisy: offsets")) != BO_OK) return s;
  if (m == 2) {
    if ((s = palloc(&sc.btmp, (size_t)S * (n + 1) * 4, st, "noisy: boxes")) != BO_OK) return s;
  } else {
    if ((s = palloc(&sc.Fd, (size_t)S * n * m, st, "noisy: in-sample draws")) != BO_OK) return s;
    if ((s = palloc(&sc.btmp, (size_t)S * (3 * n + 1) * 6, st, "noisy: boxes")) != BO_OK) return s;
  }
  if ((s = palloc(&z.Lp0, (size_t)m * M.lp_per_obj, st, "noisy: packed factor")) != BO_OK) return s;
  if ((s = palloc(&z.front, (size_t)S * n, st, "noisy: fronts")) != BO_OK) return s;

  std::vector<double> hyp(nhyp, 0.0);
  for (int i = 0; i < m * d; ++i) hyp[i] = 1.0 / static_cast<double>(M.ls[i]);
  for (int k = 0; k < m; ++k) {
    hyp[(size_t)m * d + k] = M.os[k];
    hyp[(size_t)m * d + m + k] = M.noise[k];
    if (comp) {
      hyp[(size_t)m * d + 3 * m + k] = M.s_dep[k];
      hyp[(size_t)m * d + 4 * m + k] = M.s_int[k];
    }
  }
  if (comp)
    for (size_t i = 0; i < (size_t)m * dc; ++i) hyp[(size_t)m * d + 5 * m + i] = M.prefh[i];
  // pinned staging: [hyp][flags 16 B][Y][counts][maxima][offsets]
  DeviceState* DS = device_state(M.device);
  if (!DS) return fail(BO_ERR_DEVICE, W_ + ": device index out of range");
  std::lock_guard<std::mutex> stage_lock(DS->fit_mu);
  const size_t off_flag = (sizeof(double) * nhyp + 15) / 16 * 16;
  const size_t off_stats = off_flag + 32;
  const size_t off_y = off_stats + 16 * 3;
  const size_t off_cnt = (off_y + sizeof(float) * n * m + 15) / 16 * 16;
  const size_t off_gmax = (off_cnt + sizeof(int) * 2 * S + 15) / 16 * 16;
  const size_t off_off = off_gmax + sizeof(double) * m * kAbsmaxParts;
  const size_t need = off_off + sizeof(int) * ((size_t)S + 1);
  hipError_t e = hipSuccess;
  if (need > DS->fit_stage_bytes) {
    if (DS->fit_stage) (void)hipHostFree(DS->fit_stage);
    DS->fit_stage = nullptr;
    DS->fit_stage_bytes = 0;
    const size_t cap = std::max<size_t>(need, size_t(1) << 16);
    e = hipHostMalloc(reinterpret_cast<void**>(&DS->fit_stage), cap, hipHostMallocDefault);
    if (e != hipSuccess) return hip_fail(e, "bo_nehvi_prepare: pinned staging");
    DS->fit_stage_bytes = cap;
  }
  unsigned char* stage = DS->fit_stage;
  auto sync_fail = [&](bo_status st_) {
    (void)hipStreamSynchronize(st);   // copies from the staging buffer may be pending
    if (DS->side) (void)hipStreamSynchronize(DS->side);   // and work on the side stream
    release_noisy(&M);
    return st_;
  };
  std::memcpy(stage, hyp.data(), sizeof(double) * nhyp);
  std::memcpy(stage + off_y, M.Yh.data(), sizeof(float) * n * m);
  e = hipMemcpyAsync(sc.hyp, stage, sizeof(double) * nhyp, hipMemcpyHostToDevice, st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(sc.Y, stage + off_y, sizeof(float) * n * m, hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipMemsetAsync(sc.flag, 0, 8 * sizeof(int), st);
  if (e == hipSuccess) e = hipMemsetAsync(sc.stats, 0, sizeof(unsigned long long) * 2 * m, st);
  if (e != hipSuccess) return sync_fail(hip_fail(e, "bo_nehvi_prepare: upload"));

  GramParams gp;
  gp.ils = sc.hyp;
  gp.os = sc.hyp + (size_t)m * d;
  gp.noise = gp.os + m;
  if (comp) {
    gp.dr = M.dr;
    gp.s_dep = gp.noise + 2 * m;
    gp.s_int = gp.s_dep + m;
    gp.pref = gp.s_int + m;
  }
  GramParams g0 = gp;
  g0.noise = gp.noise + m;                  // zeros: the noise-free K_XX
  auto step = [&](hipError_t err, const char* what) { return after_launch(err, st, what); };
  // The noise-free K_XX (factor, inverse, packed for the conditional
  // (co)variance) is independent of K's chain: it runs on the side stream,
  // after the uploads above, and joins before its factor is used.
  if ((s = side_stream(DS)) != BO_OK) return sync_fail(s);
  hipStream_t side = DS->side;
  auto sstep = [&](hipError_t err, const char* what) { return after_launch(err, side, what); };
  e = hipEventRecord(DS->side_evt[0], st);
  if (e == hipSuccess) e = hipStreamWaitEvent(side, DS->side_evt[0], 0);
  if (e != hipSuccess) return sync_fail(hip_fail(e, "bo_nehvi_prepare: side stream"));
  if ((s = sstep(launch_gram(M.Xd, n, d, m, nf, g0, sc.A0, side, sc.stats), "gram")) != BO_OK) return sync_fail(s);
  if ((s = sstep(launch_cholesky(sc.A0, sc.W0, nf, m, sc.flag + 2, side), "cholesky")) != BO_OK) return sync_fail(s);
  if ((s = sstep(launch_pack_factor(sc.W0, n, m, nf, M.nb, z.Lp0, sc.stats + m, sc.flag + 3, side), "pack")) != BO_OK) return sync_fail(s);
  e = hipEventRecord(DS->side_evt[1], side);
  if (e != hipSuccess) return sync_fail(hip_fail(e, "bo_nehvi_prepare: side stream"));
  // K = K_XX + eta I: factor, inverse, alpha (fp64), then K^{-1}
  if ((s = step(launch_gram(M.Xd, n, d, m, nf, gp, sc.A, st), "gram")) != BO_OK) return sync_fail(s);
  if ((s = step(launch_cholesky(sc.A, sc.W, nf, m, sc.flag, st), "cholesky")) != BO_OK) return sync_fail(s);
  if ((s = step(launch_alpha(sc.W, sc.Y, n, m, nf, M.n_pad, sc.tmp, sc.alpha, st, sc.alpha64), "alpha")) != BO_OK) return sync_fail(s);
  if ((s = step(launch_kinv(sc.A, sc.W, nf, m, st), "inverse")) != BO_OK) return sync_fail(s);
  // in-sample posterior covariance eta (I - eta K^{-1}) and its factor
  if ((s = step(launch_sigma_xx(sc.A, n, nf, m, gp.noise, st), "in-sample covariance")) != BO_OK) return sync_fail(s);
  if ((s = step(launch_cholesky(sc.A, sc.W, nf, m, sc.flag + 1, st), "cholesky")) != BO_OK) return sync_fail(s);
  // the noise-free factor from the side stream
  e = hipStreamWaitEvent(st, DS->side_evt[1], 0);
  if (e != hipSuccess) return sync_fail(hip_fail(e, "bo_nehvi_prepare: side stream"));
  // T1 = L_XX Z_X, G = K_XX^{-1} T1 = W0^T (W0 T1)
  if ((s = step(launch_gather_z(ZX, n, m, S, nf, Sp, sc.Zk, st), "gather")) != BO_OK) return sync_fail(s);
  if ((s = step(launch_trmm(false, sc.A, sc.Zk, sc.T1, nf, Sp, m, st), "trmm")) != BO_OK) return sync_fail(s);
  if ((s = step(launch_trmm(false, sc.W0, sc.T1, sc.Zk, nf, Sp, m, st), "trmm")) != BO_OK) return sync_fail(s);
  if ((s = step(launch_trmm(true, sc.W0, sc.Zk, sc.G, nf, Sp, m, st), "trmm")) != BO_OK) return sync_fail(s);
  if (m == 2) {
    // fronts and boxes of every draw on the device
    NehviFrontArgs fa;
    fa.Y = sc.Y; fa.alpha64 = sc.alpha64; fa.noise = gp.noise; fa.T1 = sc.T1;
    fa.n = n; fa.nf = nf; fa.Sp = Sp; fa.S = S;
    fa.ref0 = ref[0]; fa.ref1 = ref[1];
    fa.cons = lower != nullptr;
    fa.low0 = lower ? lower[0] : -INFINITY;
    fa.low1 = lower ? lower[1] : -INFINITY;
    fa.boxes = sc.btmp; fa.counts = sc.counts; fa.front = z.front;
    if ((s = step(launch_sample_fronts(fa, st), "fronts")) != BO_OK) return sync_fail(s);
    e = hipMemcpyAsync(stage + off_cnt, sc.counts, sizeof(int) * S, hipMemcpyDeviceToHost, st);
    if (e != hipSuccess) return sync_fail(hip_fail(e, "bo_nehvi_prepare: counts"));
  } else {
    // three objectives: the draws, then every draw's front and boxes on the device
    if ((s = step(launch_insample_values(sc.Y, sc.alpha64, gp.noise, sc.T1, n, m, nf, Sp, S, sc.Fd, st), "draws")) != BO_OK) return sync_fail(s);
    NehviFront3Args fa;
    fa.F = sc.Fd; fa.n = n; fa.S = S;
    for (int k = 0; k < 3; ++k) {
      fa.ref[k] = ref[k];
      fa.low[k] = lower ? lower[k] : -INFINITY;
    }
    fa.cons = lower != nullptr;
    fa.boxes = sc.btmp; fa.counts = sc.counts; fa.front = z.front; fa.bad = sc.flag + 4;
    if ((s = step(launch_sample_fronts3(fa, st), "fronts")) != BO_OK) return sync_fail(s);
    e = hipMemcpyAsync(stage + off_cnt, sc.counts, sizeof(int) * 2 * S, hipMemcpyDeviceToHost, st);
    if (e != hipSuccess) return sync_fail(hip_fail(e, "bo_nehvi_prepare: counts"));
  }
  if ((s = step(launch_absmax(sc.G, (int64_t)nf * Sp, m, sc.gmax, st), "absmax")) != BO_OK) return sync_fail(s);
  e = hipMemcpyAsync(stage + off_flag, sc.flag, 8 * sizeof(int), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(stage + off_stats, sc.stats, sizeof(unsigned long long) * 2 * m,
                       hipMemcpyDeviceToHost, st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(stage + off_gmax, sc.gmax, sizeof(double) * m * kAbsmaxParts,
                       hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return sync_fail(hip_fail(e, "bo_nehvi_prepare: sync"));
  int flags[8];
  std::memcpy(flags, stage + off_flag, sizeof(flags));
  if (flags[0]) return sync_fail(fail(BO_ERR_NOT_POSITIVE_DEFINITE, W_ + ": K not positive definite"));
  if (flags[1]) return sync_fail(fail(BO_ERR_NOT_POSITIVE_DEFINITE, W_ + ": in-sample posterior covariance not positive definite"));
  if (flags[2] || flags[3]) return sync_fail(fail(BO_ERR_NOT_POSITIVE_DEFINITE, W_ + ": noise-free K_XX not positive definite"));
  {
    // the conditional uses the noise-free K_XX's inverse factor: the same
    // conditioning limit as the fit's
    unsigned long long st_bits[6];
    std::memcpy(st_bits, stage + off_stats, sizeof(unsigned long long) * 2 * m);
    for (int k = 0; k < m; ++k) {
      const double kd = bits_to_double(st_bits[k]), wm = bits_to_double(st_bits[m + k]);
      const double ce = kd * wm * wm;
      if (!(ce < kCondLimit)) {
        char msg[200];
        std::snprintf(msg, sizeof msg,
                      ": objective %d: the noise-free K_XX has max K_ii * max |L^-1|^2 = %.3g, "
                      "at or above 2^24",
                      k, ce);
        return sync_fail(fail(BO_ERR_ILL_CONDITIONED, W_ + msg));
      }
    }
  }
  const int* cnt_h = reinterpret_cast<const int*>(stage + off_cnt);
  z.counts.assign(cnt_h, cnt_h + S);
  z.fsize.resize(S);
  if (m == 2) {
    for (int i = 0; i < S; ++i) z.fsize[i] = z.counts[i] - 1;     // the staircase has P + 1 boxes
  } else {
    if (flags[4]) return sync_fail(fail(BO_ERR_NONFINITE_INPUT, W_ + ": non-finite in-sample draw"));
    for (int i = 0; i < S; ++i) z.fsize[i] = cnt_h[S + i];
  }
  int* off = reinterpret_cast<int*>(stage + off_off);
  int64_t total = 0;
  for (int i = 0; i < S; ++i) {
    off[i] = static_cast<int>(total);
    total += z.counts[i];
  }
  off[S] = static_cast<int>(total);
  if (total > (int64_t)1 << 28)
    return sync_fail(fail(BO_ERR_CAPACITY, W_ + ": too many per-draw boxes"));
  if (nehvi_ehvi_lds_bytes(S, 4, m, 0, false) > kLdsLimit)
    return sync_fail(fail(BO_ERR_CAPACITY, W_ + ": base samples exceed LDS"));
  double gmax[3] = {0.0, 0.0, 0.0};
  {
    const double* parts = reinterpret_cast<const double*>(stage + off_gmax);
    for (int k = 0; k < m; ++k)
      for (int b = 0; b < kAbsmaxParts; ++b) gmax[k] = std::max(gmax[k], parts[k * kAbsmaxParts + b]);
  }
  float scale[3] = {1.f, 1.f, 1.f};
  for (int k = 0; k < m; ++k) {
    // a power of two that brings max |G| into [2^13, 2^14): the fp16 low
    // halves then stay clear of the subnormal range
    int ex = 0;
    if (gmax[k] > 0.0 && std::isfinite(gmax[k])) ex = 13 - static_cast<int>(std::floor(std::log2(gmax[k])));
    ex = std::max(-60, std::min(60, ex));
    scale[k] = std::ldexp(1.0f, ex);
    z.ginv[k] = std::ldexp(1.0f, -ex);
  }
  if ((s = palloc(&z.Gp, (size_t)m * n32 * nrb * 1024, st, "noisy: G fragments")) != BO_OK) return sync_fail(s);
  if ((s = palloc(&z.boxes, (size_t)std::max<int64_t>(total, 1) * 2 * m, st, "noisy: boxes")) != BO_OK) return sync_fail(s);
  if ((s = palloc(&z.off, (size_t)S + 1, st, "noisy: box offsets")) != BO_OK) return sync_fail(s);
  e = hipMemcpyAsync(z.off, off, sizeof(int) * (S + 1), hipMemcpyHostToDevice, st);
  if (e != hipSuccess) return sync_fail(hip_fail(e, "bo_nehvi_prepare: offsets"));
  if (m == 2) {
    if ((s = step(launch_compact_boxes(sc.btmp, (int64_t)(n + 1) * 4, z.off, S, z.boxes, st), "boxes")) != BO_OK) return sync_fail(s);
  } else {
    if ((s = step(launch_compact_boxes3(sc.btmp, (int64_t)(3 * n + 1) * 6, z.off, S, z.boxes, st), "boxes")) != BO_OK) return sync_fail(s);
  }
  if ((s = step(launch_pack_g(sc.G, nf, Sp, n32, m, scale, z.Gp, st), "pack G")) != BO_OK) return sync_fail(s);
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return sync_fail(hip_fail(e, "bo_nehvi_prepare: sync"));
  z.S = S; z.Sp = Sp; z.n32 = n32; z.total = static_cast<int>(total); z.m = m;
  z.cons = lower != nullptr;
  for (int k = 0; k < 3; ++k) z.low[k] = (lower && k < m) ? lower[k] : -INFINITY;
  return mark_call(M, st, "bo_nehvi_prepare: stream ordering");
}

bo_status score_nehvi_impl(bo_model model, const float* cand, int64_t M_, int32_t q,
                           const float* Z, int32_t S, float* ehvi, void* stream) {
  if (!model) return fail(BO_ERR_INVALID_ARGUMENT, "bo_score_nehvi: model is NULL");
  Model& M = model->m;
  Model::Noisy& z = M.nz;
  if (z.S == 0) return fail(BO_ERR_INVALID_ARGUMENT, "bo_score_nehvi: call bo_nehvi_prepare first");
  if (S != z.S) return fail(BO_ERR_INVALID_ARGUMENT, "bo_score_nehvi: S differs from the prepared S");
  if (q != 1 && q != 2 && q != 4) return fail(BO_ERR_INVALID_ARGUMENT, "bo_score_nehvi: q must be 1, 2 or 4");
  if (M_ < 0) return fail(BO_ERR_INVALID_ARGUMENT, "bo_score_nehvi: M < 0");
  if (M_ > (int64_t)1 << 40) return fail(BO_ERR_CAPACITY, "bo_score_nehvi: M too large");
  if (M_ == 0) return BO_OK;
  DeviceGuard g(M.device);
  if (!g.ok) return fail(BO_ERR_DEVICE, "bo_score_nehvi: cannot select the model's device");
  const int m = M.m;
  bo_status s;
  if ((s = check_dev(cand, sizeof(float) * M_ * q * M.d, "cand")) != BO_OK) return s;
  if ((s = check_dev(Z, sizeof(float) * (size_t)S * q * m, "base_samples")) != BO_OK) return s;
  if ((s = check_dev(ehvi, sizeof(float) * M_, "ehvi")) != BO_OK) return s;
  if (posterior_lds_bytes(M.nb, q) > kLdsLimit)
    return fail(BO_ERR_CAPACITY, "bo_score_nehvi: posterior tile exceeds LDS");
  if (nehvi_ehvi_lds_bytes(S, q, m, 0, false) > kLdsLimit)
    return fail(BO_ERR_CAPACITY, "bo_score_nehvi: base samples exceed LDS");
  hipStream_t st = static_cast<hipStream_t>(stream);
  if ((s = order_after_previous(M, st, "bo_score_nehvi: stream ordering")) != BO_OK) return s;
  const int T = q * (q + 1) / 2;
  const int64_t Cb = std::min<int64_t>(M_, kNehviChunk / q);   // batches per chunk
  const int64_t C = Cb * q;                                     // points per chunk
  const size_t need = 2 * (size_t)C * m + (q > 1 ? (size_t)Cb * m * T : 0) +
                      (size_t)m * S * C;
  if (need > z.ws_floats) {
    if (z.ws) {
      hipError_t e = hipDeviceSynchronize();      // earlier launches may use it
      if (e != hipSuccess) return hip_fail(e, "bo_score_nehvi: sync before workspace growth");
      pfree(z.ws, st);
    }
    z.ws_floats = 0;
    if ((s = palloc(&z.ws, need, st, "noisy: scoring workspace")) != BO_OK) return s;
    z.ws_floats = need;
  }
  // planar per objective: each posterior launch writes whole cache lines
  float* mu_buf = z.ws;                                          // [m][C]
  float* sd_buf = z.ws + (size_t)C * m;                          // [m][C] marginal tau
  float* ch_buf = sd_buf + (size_t)C * m;                        // q > 1: [m][Cb][T] factors
  float* dbuf = ch_buf + (q > 1 ? (size_t)Cb * m * T : 0);       // [m][S][C]
  for (int64_t b0 = 0; b0 < M_; b0 += Cb) {
    const int64_t nb_ = std::min<int64_t>(Cb, M_ - b0);
    const int64_t np_ = nb_ * q;
    const float* cc = cand + b0 * q * M.d;
    for (int k = 0; k < m; ++k) {
      PosteriorArgs pa = posterior_args(M, k, z.Lp0, cc, np_, q);
      // chunk-sized planes: the EHVI kernel reads them at the chunk's nbat
      pa.mu = mu_buf + (size_t)k * np_; pa.sd = sd_buf + (size_t)k * np_;
      pa.mu_ps = pa.sd_ps = 1;
      pa.chol = (q > 1) ? ch_buf + (size_t)k * nb_ * T : nullptr;
      if ((s = after_launch(launch_posterior(pa, st), st, "posterior")) != BO_OK) return s;
    }
    NehviMeansArgs ma;
    ma.cand = cc; ma.npts = np_; ma.d = M.d; ma.dx = M.dx; ma.n32 = z.n32;
    ma.n_pad = M.n_pad; ma.S = S; ma.Xs = M.Xs; ma.invls = M.invls; ma.Gp = z.Gp;
    ma.xf = M.xf; ma.xf_stride = (int64_t)M.nb * dist_frags(M.dx) * 512;
    ma.x2 = M.x2; ma.ctr = M.ctr;
    for (int k = 0; k < 3; ++k) {
      ma.s[k] = k < m ? M.os[k] : 0.f;
      ma.kbound[k] = k < m ? M.kbound[k] : 1.f;
      ma.ginv[k] = z.ginv[k];
      ma.s_dep[k] = (M.dr > 0 && k < m) ? M.s_dep[k] : 0.f;
      ma.s_int[k] = (M.dr > 0 && k < m) ? M.s_int[k] : 0.f;
    }
    ma.dr = M.dr; ma.dr4 = M.dr4; ma.wts = M.wts; ma.pref = M.pref;
    ma.out = dbuf; ma.ldo = C;
    if ((s = after_launch(launch_nehvi_means(ma, m, st), st, "conditional means")) != BO_OK) return s;
    NehviEhviArgs ea;
    ea.mu = mu_buf; ea.sd = sd_buf; ea.chol = ch_buf; ea.D = dbuf; ea.ldd = C; ea.Z = Z;
    ea.boxes = z.boxes; ea.off = z.off; ea.total = z.total; ea.nbat = nb_; ea.S = S;
    ea.q = q; ea.m = m; ea.cons = z.cons;
    for (int k = 0; k < 3; ++k) ea.low[k] = z.low[k];
    ea.ehvi = ehvi + b0;
    if ((s = after_launch(launch_nehvi_ehvi(ea, st), st, "noisy ehvi")) != BO_OK) return s;
  }
  z.q = q;
  return mark_call(M, st, "bo_score_nehvi: stream ordering");
}

}  // namespace

extern "C" {

bo_status bo_nehvi_prepare(bo_model model, const float* base_samples_X, int32_t S,
                           const float* ref_point, const float* feas_lower, void* stream) {
  return nehvi_prepare_impl(model, base_samples_X, S, ref_point, feas_lower, stream);
}

bo_status bo_score_nehvi(bo_model model, const float* cand, int64_t M, int32_t q,
                         const float* base_samples, int32_t S, float* ehvi, void* stream) {
  return score_nehvi_impl(model, cand, M, q, base_samples, S, ehvi, stream);
}

bo_status bo_nehvi_front(bo_model model, int32_t sample, int32_t* idx_host, int32_t cap,
                         int32_t* count) {
  if (!model || !count || cap < 0 || (cap > 0 && !idx_host))
    return fail(BO_ERR_INVALID_ARGUMENT, "bo_nehvi_front: bad argument");
  Model& M = model->m;
  if (M.nz.S == 0) return fail(BO_ERR_INVALID_ARGUMENT, "bo_nehvi_front: not prepared");
  if (sample < 0 || sample >= M.nz.S)
    return fail(BO_ERR_INVALID_ARGUMENT, "bo_nehvi_front: sample out of range");
  const int32_t P = M.nz.fsize[sample];
  *count = P;
  const int32_t k = std::min(cap, P);
  if (k > 0) {
    DeviceGuard g(M.device);
    hipError_t e = hipMemcpy(idx_host, M.nz.front + (size_t)sample * M.n, sizeof(int32_t) * k,
                             hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "bo_nehvi_front: copy");
  }
  return BO_OK;
}

bo_status bo_profile_enable(int32_t on) {
  Profile& P = profile();
  std::lock_guard<std::mutex> lk(P.mu);
  if (on && P.pool.empty()) {
    P.pool.resize(kProfileCap);
    for (auto& r : P.pool)
      for (auto& e : r.e) {
        hipError_t err = hipEventCreate(&e);
        if (err != hipSuccess) return hip_fail(err, "bo_profile_enable");
      }
  }
  P.on = on != 0;
  P.used = 0;
  return BO_OK;
}

bo_status bo_profile_read(double* posterior_ms, double* ehvi_ms, int64_t* calls,
                          int64_t* posterior_launches) {
  if (!posterior_ms || !ehvi_ms || !calls || !posterior_launches)
    return fail(BO_ERR_INVALID_ARGUMENT, "bo_profile_read: NULL output");
  Profile& P = profile();
  std::lock_guard<std::mutex> lk(P.mu);
  double a = 0.0, b = 0.0;
  int64_t launches = 0;
  for (size_t i = 0; i < P.used; ++i) {
    Profile::Rec& r = P.pool[i];
    hipError_t e = hipEventSynchronize(r.e[2]);
    float t01 = 0.f, t12 = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&t01, r.e[0], r.e[1]);
    if (e == hipSuccess) e = hipEventElapsedTime(&t12, r.e[1], r.e[2]);
    if (e != hipSuccess) return hip_fail(e, "bo_profile_read");
    a += t01;
    b += t12;
    launches += r.launches;
  }
  *posterior_ms = a;
  *ehvi_ms = b;
  *calls = static_cast<int64_t>(P.used);
  *posterior_launches = launches;
  P.used = 0;
  return BO_OK;
}

bo_status bo_argmax(const float* values, int64_t M, int64_t* index, float* value, void* stream) {
  if (M < 0 || M >= ((int64_t)1 << 31)) return fail(BO_ERR_INVALID_ARGUMENT, "bo_argmax: M out of range");
  bo_status s;
  if ((s = check_dev(index, sizeof(int64_t), "index")) != BO_OK) return s;
  if ((s = check_dev(value, sizeof(float), "value")) != BO_OK) return s;
  if (M > 0 && (s = check_dev(values, sizeof(float) * M, "values")) != BO_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  return after_launch(launch_argmax(values, M, index, value, st), st, "argmax");
}

bo_status bo_measure_peak(int32_t what, int64_t iters, double* rate, void* stream) {
  if (!rate || what < BO_PEAK_VALU_FMA || what > BO_PEAK_MFMA_F16 || iters < 1 || iters > (1 << 24))
    return fail(BO_ERR_INVALID_ARGUMENT, "bo_measure_peak: bad argument");
  hipError_t e = measure_peak(what, iters, rate, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "bo_measure_peak");
  return BO_OK;
}

bo_status bo_draw_fronts3_test(const double* F, int64_t n, int32_t S, const float* ref,
                               const float* feas_lower, int32_t* front, float* boxes,
                               int32_t* counts, void* stream) {
  const std::string W("bo_draw_fronts3_test");
  if (n < 1 || S < 1) return fail(BO_ERR_INVALID_ARGUMENT, W + ": n < 1 or S < 1");
  if (n > BO_MAX_N) return fail(BO_ERR_CAPACITY, W + ": n beyond limit");
  if (!ref) return fail(BO_ERR_INVALID_ARGUMENT, W + ": ref is NULL");
  if (!all_finite(ref, 3)) return fail(BO_ERR_NONFINITE_INPUT, W + ": ref not finite");
  if (feas_lower)
    for (int k = 0; k < 3; ++k)
      if (std::isnan(feas_lower[k])) return fail(BO_ERR_NONFINITE_INPUT, W + ": threshold is NaN");
  if (nehvi_front3_lds_bytes(n) > kLdsLimit) return fail(BO_ERR_CAPACITY, W + ": n beyond LDS");
  bo_status s;
  if ((s = check_dev(F, sizeof(double) * (size_t)S * n * 3, "F")) != BO_OK) return s;
  if ((s = check_dev(front, sizeof(int32_t) * (size_t)S * n, "front")) != BO_OK) return s;
  if ((s = check_dev(boxes, sizeof(float) * (size_t)S * (3 * n + 1) * 6, "boxes")) != BO_OK) return s;
  if ((s = check_dev(counts, sizeof(int32_t) * 2 * (size_t)S, "counts")) != BO_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  int* bad = nullptr;
  if ((s = palloc(&bad, 1, st, "flag")) != BO_OK) return s;
  hipError_t e = hipMemsetAsync(bad, 0, sizeof(int), st);
  NehviFront3Args fa;
  fa.F = F; fa.n = n; fa.S = S;
  for (int k = 0; k < 3; ++k) {
    fa.ref[k] = ref[k];
    fa.low[k] = feas_lower ? feas_lower[k] : -INFINITY;
  }
  fa.cons = feas_lower != nullptr;
  fa.boxes = boxes; fa.counts = counts; fa.front = front; fa.bad = bad;
  if (e == hipSuccess) e = launch_sample_fronts3(fa, st);
  int flag = 0;
  if (e == hipSuccess) e = hipMemcpyAsync(&flag, bad, sizeof(int), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  pfree(bad, st);
  if (e != hipSuccess) return hip_fail(e, "bo_draw_fronts3_test: launch");
  if (flag) return fail(BO_ERR_NONFINITE_INPUT, W + ": non-finite value");
  return BO_OK;
}

bo_status bo_cholesky_test(const float* A, int64_t n, float* L, void* stream) {
  if (n < 1) return fail(BO_ERR_INVALID_ARGUMENT, "bo_cholesky_test: n < 1");
  if (n > BO_MAX_N) return fail(BO_ERR_CAPACITY, "bo_cholesky_test: n beyond limit");
  bo_status s;
  if ((s = check_dev(A, sizeof(float) * n * n, "A")) != BO_OK) return s;
  if ((s = check_dev(L, sizeof(float) * n * n, "L")) != BO_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int nf = static_cast<int>((n + kFitBlk - 1) / kFitBlk) * kFitBlk;
  FitScratch fs;
  fs.st = st;
  fs.own = true;
  if ((s = palloc(&fs.A, (size_t)nf * nf, st, "matrix")) != BO_OK) return s;
  if ((s = palloc(&fs.W, (size_t)nf * nf, st, "inverse")) != BO_OK) return s;
  if ((s = palloc(&fs.flag, 1, st, "flag")) != BO_OK) return s;
  hipError_t e = hipMemsetAsync(fs.flag, 0, sizeof(int), st);
  if (e != hipSuccess) return hip_fail(e, "bo_cholesky_test: memset");
  if ((s = after_launch(launch_f32_to_padded(A, n, nf, fs.A, st), st, "pad")) != BO_OK) return s;
  if ((s = after_launch(launch_cholesky(fs.A, fs.W, nf, 1, fs.flag, st), st, "cholesky")) != BO_OK) return s;
  if ((s = after_launch(launch_lower_to_f32(fs.A, n, nf, L, st), st, "convert")) != BO_OK) return s;
  int flag = 0;
  e = hipMemcpyAsync(&flag, fs.flag, sizeof(int), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "bo_cholesky_test: sync");
  if (flag) return fail(BO_ERR_NOT_POSITIVE_DEFINITE, "bo_cholesky_test: non-positive pivot");
  return BO_OK;
}

}  // extern "C"
