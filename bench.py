#!/usr/bin/env python3
"""Benchmark: candidates scored per second on one MI355X.

Workload: 1,048,576 encoded candidates, n = 1024 observations, d = 16,
m = 2 objectives, q = 1, S = 512 Monte-Carlo samples (the headline
configuration), seeded synthetic inputs resident in HBM before timing.

One step = one pass of the acquisition hot path over the whole batch:
bo_score (posterior + MC-EHVI of every candidate, mu/sigma not materialised)
+ bo_argmax, on a model fitted once before timing (bo_fit is timed apart and
reported in phases_ms). W warm-up steps, then K timed steps, each bracketed by
HIP events on the stream the library launches on; value = M / (median step
time). The K steps are also timed on the host between device
synchronisations (ms_per_step_wall).

The JSON line also carries
  roofline     — the dominant kernel, the posterior (cross-covariance plus
                 the triangular L^{-1} K*^T product, on the fp16 matrix cores
                 as three products of power-of-two-scaled fp16 hi/lo operand
                 halves with fp32 accumulation): its algorithmic flops per
                 launch, each multiply-add of the triangle counted once
                 (n^2 + 2nd + 2n + 2n per point), over its mean launch time
                 from HIP events recorded on its stream during the timed steps,
                 against the dense fp16 MFMA peak (the dtype the matrix cores
                 execute); the issued split-product rate is reported beside it;
  cpu_baseline — the fp64 oracle timed on this host's cores (candidate tiles
                 spread over a process pool forked before the GPU is touched)
                 on a bounded sample of the same candidates (score + argmax;
                 its fit is timed apart).
"""
from __future__ import annotations

import argparse
import json
import multiprocessing
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_FP16_MFMA_TFLOPS = 2500.0   # dense (no 2:1 sparsity)
PEAK_FP64_MFMA_TFLOPS = 78.6
# VALU issue peak derived from the unit counts: 256 CUs x 128 fp32 lanes per
# clock (the 157.3 TFLOP/s vector figure counted as 2 flops per FMA lane-op)
# x 2.4 GHz.
PEAK_VALU_LANE_OPS = 256 * 128 * 2.4e9
METRIC = "candidates scored/sec (GP posterior + MC-EHVI), n=1024 d=16 S=512, 1 GPU"


def posterior_f16_mfma_flops_per_point(n: int, d: int) -> float:
    """fp16 MFMA flops issued per point for one objective: the triangle's
    n(n+1)/2 multiply-adds as three split products (hi*hi, hi*lo, lo*hi), plus
    the distance dot products (hi and scaled-lo streams over 2d positions,
    padded to 32-wide MFMA k-steps)."""
    kpos = 32 * ((d + 31) // 32 + (2 * d + 31) // 32)
    return 3.0 * n * (n + 1) + 2.0 * n * kpos


def posterior_flops_per_point(n: int, d: int, q: int) -> float:
    """Algorithmic flops of one point's posterior for one objective, each
    multiply-add counted once: n^2 for the lower-triangular product
    L^{-1} k* (n(n+1)/2 multiply-adds, counted as n^2), 2nd for the scaled
    distances, 2n for mu = k*^T alpha and 2n for |v|^2 (q = 1) or
    2n(q+1)/2 per point for the batch V^T V."""
    return n * n + 2.0 * n * d + 2.0 * n + 2.0 * n * (q + 1) / 2.0


def ehvi_lane_ops(M: int, q: int, m: int, S: int, nbox: int) -> float:
    """Algorithmic VALU work of the MC-EHVI in lane-operations, counting a
    multiply-add as one: per (candidate, sample, box) a subtraction and a clamp
    per objective and member, for q > 1 the running minima of the 2^q - 1
    member subsets, and m - 1 multiplies per subset (the last one fused with
    the accumulation); per (candidate, sample) the reparameterised draw
    (m FMAs for q = 1, m q(q+1)/2 for the lower-factor product)."""
    subsets = 2 ** q - 1
    per_box = 2 * q * m + (subsets - q) * m + subsets * (m - 1)
    draw = m if q == 1 else m * q * (q + 1) // 2
    return float(M) * S * (nbox * per_box + draw)


def recorded_traffic(n_launch_flops_workload: str):
    """HBM bytes per posterior launch from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, copy-calibrated), or None when the kernel source
    has changed since those counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "posterior_counters.json")
    try:
        rec = json.load(open(path))
        src = open(os.path.join(ROOT, rec["source"]), "rb").read()
    except (OSError, ValueError, KeyError):
        return None
    if hashlib.sha256(src).hexdigest() != rec.get("source_sha256"):
        return None
    if rec.get("workload", "").split(" ")[0] != n_launch_flops_workload:
        return None
    return rec["traffic_bytes_per_launch"]


def host_info():
    """The host the CPU baseline runs on: CPU model and sockets (from
    /proc/cpuinfo), core counts, the BLAS numpy uses and its thread settings."""
    info = {"os_cpu_count": os.cpu_count()}
    try:
        info["affinity_cpus"] = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        info["affinity_cpus"] = os.cpu_count()
    models, sockets = set(), set()
    try:
        for line in open("/proc/cpuinfo"):
            key, _, val = line.partition(":")
            key = key.strip()
            if key == "model name":
                models.add(val.strip())
            elif key == "physical id":
                sockets.add(val.strip())
    except OSError:
        pass
    info["cpu_model"] = "; ".join(sorted(models)) or None
    info["sockets"] = len(sockets) or None
    try:
        blas = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        info["blas"] = f"{blas.get('name')} {blas.get('version')}"
    except Exception:  # pragma: no cover
        info["blas"] = None
    info["thread_env"] = {k: os.environ.get(k) for k in
                          ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")}
    return info


_POOL = {}


def _oracle_tile(bounds):
    """One tile of the CPU baseline in a pool worker: the oracle's score of
    candidates [i0, i1) with one BLAS thread (the pool spreads the tiles)."""
    import oracle as O
    from threadpoolctl import threadpool_limits
    i0, i1 = bounds
    with threadpool_limits(1):
        out = O.score(_POOL["model"], _POOL["cand"][i0:i1], _POOL["ref"], _POOL["Z"])
    return out["ehvi"]


def cpu_baseline(wl, sample: int, workers: int, tile: int = 1024):
    """The fp64 oracle (score + argmax) on the first ``sample`` candidates,
    tiles of ``tile`` candidates spread over ``workers`` forked processes with
    one BLAS thread each. Must run before the GPU is initialised (the pool is
    forked from this process)."""
    import oracle as O
    t0 = time.perf_counter()
    model = O.fit(wl.X, wl.Y, wl.lengthscale, wl.outputscale, wl.noise)
    fit_s = time.perf_counter() - t0
    _POOL.update(model=model, cand=wl.cand[:sample].astype(np.float64), ref=wl.ref,
                 Z=wl.Z.astype(np.float64))
    tiles = [(i, min(i + tile, sample)) for i in range(0, sample, tile)]
    ctx = multiprocessing.get_context("fork")
    with ctx.Pool(workers) as pool:
        pool.map(_oracle_tile, [(0, 1)] * workers)          # workers up
        t1 = time.perf_counter()
        parts = pool.map(_oracle_tile, tiles, chunksize=1)
        O.argmax(np.concatenate(parts))
        t2 = time.perf_counter()
    _POOL.clear()
    return {
        "value": sample / (t2 - t1),
        "unit": "candidates/s",
        "cores": int(workers),
        "kind": "oracle",
        "sample": f"first {sample} candidates of the same workload in tiles of {tile} over "
                  f"{workers} processes (one BLAS thread each); fp64 oracle score + argmax "
                  f"took {t2 - t1:.2f} s (fit {fit_s:.2f} s, excluded)",
        "host": host_info(),
    }


def baseline_workers():
    """Processes for the CPU baseline: the host's CPU share (affinity),
    capped at 16 and at OMP_NUM_THREADS when it is set."""
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    cap = 16
    env = os.environ.get("OMP_NUM_THREADS")
    if env and env.isdigit() and int(env) > 0:
        cap = min(cap, int(env))
    return max(1, min(n, cap))


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-sample", type=int, default=1 << 20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-peaks", action="store_true", help="skip the achieved-peak probes")
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="also run one plain device copy of this many MiB (counter calibration)")
    a = ap.parse_args(argv)

    if a.gpus != 1:
        print(json.dumps({"error": "the scoring path runs on one GPU; --gpus must be 1 (sharding by candidates across GPUs is not built)"}))
        return 2

    import bo_inputs as bi

    wl = bi.make_config(a.config, seed=a.seed)
    # the CPU baseline forks its process pool before anything touches the GPU
    cpu = None
    if not a.no_cpu_baseline:
        cpu = cpu_baseline(wl, min(a.cpu_sample, wl.M), baseline_workers())

    import torch
    import paper_2602_10729_amd as bo

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    X = torch.from_numpy(wl.X).to(dev)
    Y = torch.from_numpy(wl.Y).to(dev)
    cand = torch.from_numpy(wl.cand).to(dev)
    Z = torch.from_numpy(wl.Z).to(dev)
    ehvi = torch.empty(wl.M, dtype=torch.float32, device=dev)
    idx = torch.empty(1, dtype=torch.int64, device=dev)
    val = torch.empty(1, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    # bo_fit (synchronous), off the step: median of five after two warm-ups
    fit_ms = []
    for i in range(7):
        t0 = time.perf_counter()
        model = bo.fit(X, Y, wl.lengthscale, wl.outputscale, wl.noise, stream=stream)
        if i >= 2:
            fit_ms.append((time.perf_counter() - t0) * 1e3)
    fit_ms = statistics.median(fit_ms)

    def step():
        bo.score(model, cand, wl.ref, Z, ehvi=ehvi, stream=stream)
        bo.argmax(ehvi, index=idx, value=val, stream=stream)

    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()

    if a.calib_copy_mb > 0:
        nbytes = a.calib_copy_mb << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # K timed steps: HIP events around each on the launch stream, the
    # library's own events around its posterior and EHVI launches, and the
    # host clock around all K between device synchronisations
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(a.steps)]
    bo.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in ev:
        e0.record(stream)
        step()
        e1.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    post_ms, ehvi_ms, calls, launches = bo.profile_read()
    bo.profile_enable(False)
    best = int(idx.item())
    step_ms = [e0.elapsed_time(e1) for e0, e1 in ev]

    ms_med = statistics.median(step_ms)
    wall_ms = (t1 - t0) * 1e3 / a.steps
    value = wl.M / (ms_med / 1e3)
    n_pts = wl.M * wl.q
    flops_launch = n_pts * posterior_flops_per_point(wl.n, wl.d, wl.q)
    issued_launch = n_pts * posterior_f16_mfma_flops_per_point(wl.n, wl.d)
    launch_ms = post_ms / max(launches, 1)
    achieved = flops_launch / (launch_ms / 1e3) / 1e12
    issued = issued_launch / (launch_ms / 1e3) / 1e12

    rec = {
        "metric": METRIC,
        "value": value,
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": ms_med,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32-class: fp32 VALU; the posterior contraction and distance dot products "
                 "on fp16 MFMA as three products of power-of-two-scaled fp16 hi/lo halves "
                 "with fp32 accumulation",
        "data": "synthetic",
        "config": {
            "workload": f"config {a.config}: M={wl.M} candidates (q={wl.q}), n={wl.n} "
                        f"observations, d={wl.d}, m={wl.m} objectives, S={wl.S} MC samples, seed {a.seed}",
            "M": wl.M, "q": wl.q, "n": wl.n, "d": wl.d, "m": wl.m, "S": wl.S,
            "step": "bo_score + bo_argmax over all M candidates (model fitted once, "
                    "bo_fit timed apart in phases_ms.fit)",
        },
        "step_ms": {"median": ms_med, "min": min(step_ms), "mean": statistics.mean(step_ms),
                    "max": max(step_ms), "timing": "HIP events on the launch stream"},
        "ms_per_step_wall": wall_ms,
        "roofline": {
            "bound": "mfma",
            "kernel": "k_posterior (one launch per objective)",
            "mfma_dtype": "f16 (three split products per multiply-add, fp32 accumulate)",
            "achieved": achieved,
            "peak": PEAK_FP16_MFMA_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_FP16_MFMA_TFLOPS,
            "traffic": recorded_traffic("headline") if a.config == 3 else None,
            "launch_ms": launch_ms,
            "flops_per_launch": flops_launch,
            "flops_formula": "M q (n^2 + 2nd + 2n + 2n(q+1)/2), each multiply-add counted once",
            "issued_mfma": {"flops_per_launch": issued_launch, "achieved": issued,
                            "frac_of_fp16_peak": issued / PEAK_FP16_MFMA_TFLOPS,
                            "formula": "M q (3 n(n+1) + 2 n 32 ceil-k-steps(3d)): the split "
                                       "products of the triangle and the distance MFMAs"},
        },
        "phases_ms": {"fit": fit_ms, "posterior_per_call": post_ms / max(calls, 1),
                      "ehvi_per_call": ehvi_ms / max(calls, 1)},
        "argmax_index": best,
    }
    nbox = len(bo.box_decomposition(wl.Y[bo.pareto_front(wl.Y, wl.ref)], wl.ref)[0])
    ehvi_ops = ehvi_lane_ops(wl.M, wl.q, wl.m, wl.S, nbox)
    ehvi_launch_ms = ehvi_ms / max(calls, 1)
    ehvi_rate = ehvi_ops / (ehvi_launch_ms / 1e3)
    rec["ehvi_roofline"] = {
        "bound": "alu", "kernel": "k_ehvi (one launch per call)", "boxes": nbox,
        "note": None if wl.q == 1 else "q > 1: boxes that add zero on a whole wave are skipped, "
                                       "so the algorithmic rate can exceed the issue peak",
        "achieved": ehvi_rate / 1e12, "peak": PEAK_VALU_LANE_OPS / 1e12,
        "unit": "T lane-ops/s", "frac": ehvi_rate / PEAK_VALU_LANE_OPS,
        "launch_ms": ehvi_launch_ms, "lane_ops_per_launch": ehvi_ops,
    }
    # the constrained acquisition (feasibility factor): same scoring calls with
    # per-objective lower bounds at the 30% quantile of the observations
    lower = bi.feasibility_thresholds(wl, 0.3)
    models_c = model
    bo.score(models_c, cand, wl.ref, Z, ehvi=ehvi, stream=stream, lower=lower)
    torch.cuda.synchronize()
    bo.profile_enable(True)
    for _ in range(a.steps):
        bo.score(models_c, cand, wl.ref, Z, ehvi=ehvi, stream=stream, lower=lower)
    torch.cuda.synchronize()
    _, cehvi_ms, ccalls, _ = bo.profile_read()
    bo.profile_enable(False)
    c_ops = ehvi_lane_ops(wl.M, wl.q, wl.m, wl.S, nbox) + float(wl.M) * wl.q * wl.S * (wl.m + 1)
    c_ms = cehvi_ms / max(ccalls, 1)
    rec["constrained_ehvi"] = {
        "bound": "alu", "kernel": "k_ehvi with feasibility weights", "lower": lower.tolist(),
        "achieved": c_ops / (c_ms / 1e3) / 1e12, "peak": PEAK_VALU_LANE_OPS / 1e12,
        "unit": "T lane-ops/s", "frac": c_ops / (c_ms / 1e3) / PEAK_VALU_LANE_OPS,
        "launch_ms": c_ms, "lane_ops_per_launch": c_ops,
    }
    # the paper's composite surrogate (routing Matern-5/2 + preference-weighted
    # deployment Matern-3/2 + interaction)
    if True:
        comp = bi.composite_hyperparameters(wl)
        t0 = time.perf_counter()
        mc = bo.fit_composite(X, Y, comp.d_route, wl.lengthscale, comp.s_route, comp.s_dep,
                              comp.s_int, comp.pref, wl.noise, stream=stream)
        cfit_ms = (time.perf_counter() - t0) * 1e3
        bo.score(mc, cand, wl.ref, Z, ehvi=ehvi, stream=stream)
        torch.cuda.synchronize()
        bo.profile_enable(True)
        for _ in range(a.steps):
            bo.score(mc, cand, wl.ref, Z, ehvi=ehvi, stream=stream)
        torch.cuda.synchronize()
        cpost_ms, _, cc, cl = bo.profile_read()
        bo.profile_enable(False)
        del mc
        c_launch = cpost_ms / max(cl, 1)
        rec["composite_posterior"] = {
            "bound": "mfma", "kernel": "k_posterior, composite kernel (one launch per objective)",
            "d_route": comp.d_route, "fit_ms": cfit_ms, "launch_ms": c_launch,
            "achieved": flops_launch / (c_launch / 1e3) / 1e12, "peak": PEAK_FP16_MFMA_TFLOPS,
            "unit": "TFLOP/s", "frac": flops_launch / (c_launch / 1e3) / 1e12 / PEAK_FP16_MFMA_TFLOPS,
            "flops": "as the roofline (triangle counted once)",
            "score_candidates_per_s": wl.M / ((cpost_ms / max(cc, 1) + ehvi_launch_ms) / 1e3),
        }
    # fp64 scoring (bo_fit_f64): the same scoring calls with the posterior in
    # double precision on the fp64 matrix cores
    mf = bo.fit(X, Y, wl.lengthscale, wl.outputscale, wl.noise, stream=stream, f64=True)
    bo.score(mf, cand, wl.ref, Z, ehvi=ehvi, stream=stream)
    torch.cuda.synchronize()
    bo.profile_enable(True)
    fsteps = max(1, min(a.steps, 5))
    for _ in range(fsteps):
        bo.score(mf, cand, wl.ref, Z, ehvi=ehvi, stream=stream)
    torch.cuda.synchronize()
    fpost_ms, fehvi_ms, fc, fl = bo.profile_read()
    bo.profile_enable(False)
    del mf
    f_launch = fpost_ms / max(fl, 1)
    rec["f64_posterior"] = {
        "bound": "mfma", "kernel": "k_posterior_f64 (one launch per objective)",
        "launch_ms": f_launch, "achieved": flops_launch / (f_launch / 1e3) / 1e12,
        "peak": PEAK_FP64_MFMA_TFLOPS, "unit": "TFLOP/s",
        "frac": flops_launch / (f_launch / 1e3) / 1e12 / PEAK_FP64_MFMA_TFLOPS,
        "score_candidates_per_s": wl.M / ((fpost_ms + fehvi_ms) / max(fc, 1) / 1e3),
    }
    # the noisy acquisition (qNEHVI): in-sample draws and per-draw fronts
    # prepared once, then whole-workload scoring calls
    if wl.m in (2, 3):
        ZX = torch.from_numpy(bi.insample_base_samples(wl)).to(dev)
        mn = bo.fit(X, Y, wl.lengthscale, wl.outputscale, wl.noise, stream=stream)
        torch.cuda.synchronize()
        # the first call also allocates its scratch in the pool and creates
        # the side stream; the figure is the median of the three calls after it
        prep = []
        for _ in range(4):
            t0 = time.perf_counter()
            bo.nehvi_prepare(mn, ZX, wl.ref, stream=stream)
            prep.append((time.perf_counter() - t0) * 1e3)
        prep_first_ms, prep_ms = prep[0], float(np.median(prep[1:]))
        bo.score_nehvi(mn, cand, Z, ehvi=ehvi, stream=stream)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(a.steps):
            bo.score_nehvi(mn, cand, Z, ehvi=ehvi, stream=stream)
        torch.cuda.synchronize()
        nz_ms = (time.perf_counter() - t0) * 1e3 / a.steps
        fronts = [len(mn.nehvi_front(s)) for s in range(0, wl.S, max(1, wl.S // 64))]
        del mn, ZX
        sp = (wl.S + 127) // 128 * 128
        rows = (wl.n + 31) // 32 * 32
        rec["noisy_acquisition"] = {
            "kernels": "k_posterior (noise-free factor) per objective, k_nehvi_means, "
                       "k_nehvi_ehvi per 1048576-point chunk",
            "prepare_ms": prep_ms, "prepare_first_call_ms": prep_first_ms, "score_ms": nz_ms,
            "batches_per_s": wl.M / (nz_ms / 1e3),
            "mean_front_size": float(np.mean(fronts)),
            "means_f16_mfma_flops_per_call": 2.0 * 3 * wl.M * wl.q * rows * sp * wl.m,
        }
    # hyperparameter fit: one exact log marginal likelihood + gradient
    # evaluation (synchronous), the unit of work of the host optimiser's loop
    bo.mll(X, Y, wl.lengthscale, wl.outputscale, wl.noise, stream=stream)
    t0 = time.perf_counter()
    reps = 5
    for _ in range(reps):
        bo.mll(X, Y, wl.lengthscale, wl.outputscale, wl.noise, stream=stream)
    mll_ms = (time.perf_counter() - t0) * 1e3 / reps
    n3 = float(wl.n) ** 3
    rec["mll"] = {
        "ms_per_evaluation": mll_ms, "evaluations_per_s": 1e3 / mll_ms,
        "gradient_entries": wl.m * (wl.d + 2),
        "fp64_flops": wl.m * (n3 / 3 + n3 / 3 + n3 / 3),
        "note": "fp64: factor n^3/3 + carried inverse n^3/3 + K^-1 = W^T W n^3/3 per objective",
    }
    if not a.no_peaks:
        rec["measured_peaks"] = {
            "valu_fma_lane_ops_per_s": bo.measure_peak(bo.PEAK_VALU_FMA, 65536),
            "valu_clamp_lane_ops_per_s": bo.measure_peak(bo.PEAK_VALU_CLAMP, 32768),
            "mfma_f32_flop_per_s": bo.measure_peak(bo.PEAK_MFMA_F32, 16384),
            "mfma_f16_flop_per_s": bo.measure_peak(bo.PEAK_MFMA_F16, 16384),
            "hbm_copy_bytes_per_s": bo.measure_peak(bo.PEAK_HBM_COPY, 1),
        }
    if cpu is not None:
        rec["cpu_baseline"] = cpu
    print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
