#!/usr/bin/env python3
"""Benchmark: candidates scored per second on one MI355X.

Workload: 1,048,576 encoded candidates, n = 1024 observations, d = 16,
m = 2 objectives, q = 1, S = 512 Monte-Carlo samples (the headline
configuration), seeded synthetic inputs resident in HBM before timing.

One step = one pass of the whole acquisition hot path over the batch:
bo_fit (GP conditioning, synchronous) + bo_score (posterior + MC-EHVI of
every candidate) + bo_argmax. W warm-up steps, then K timed steps between
device synchronisations. value = M / (seconds per step).

The JSON line also carries
  roofline     — the dominant kernel (the posterior: cross-covariance plus the
                 triangular L^{-1} K*^T product, which runs on the fp16
                 matrix cores as three products of fp16 hi/lo operand halves
                 with fp32 accumulation): the algorithmic fp16 MFMA flops per
                 launch (3 n(n+1) per point) / its mean launch time from HIP
                 events recorded on its stream during the timed steps,
                 against the MI355X dense fp16 MFMA peak; the same triangle
                 counted once (fp32-equivalent) is reported beside it against
                 the dense fp32 MFMA peak;
  cpu_baseline — the fp64 oracle timed on this host on a bounded sample of the
                 same candidates (score + argmax; its fit is timed apart).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_FP16_MFMA_TFLOPS = 2500.0   # dense (no 2:1 sparsity)
# VALU issue peak derived from the unit counts: 256 CUs x 128 fp32 lanes per
# clock (the 157.3 TFLOP/s vector figure counted as 2 flops per FMA lane-op)
# x 2.4 GHz.
PEAK_VALU_LANE_OPS = 256 * 128 * 2.4e9
METRIC = "candidates scored/sec (GP posterior + MC-EHVI), n=1024 d=16 S=512, 1 GPU"


def posterior_f16_mfma_flops_per_point(n: int) -> float:
    """fp16 MFMA flops of one point's triangular product L^{-1} k*: n(n+1)/2
    multiply-adds, each done as three split products (hi*hi, hi*lo, lo*hi)."""
    return 3.0 * n * (n + 1)


def posterior_flops_per_point(n: int, d: int, q: int) -> float:
    """Algorithmic flops of one point's posterior for one objective:
    n^2 for the lower-triangular product L^{-1} k* (n(n+1)/2 multiply-adds,
    counted as n^2), 2nd for the scaled distances, 2n for mu = k*^T alpha and
    2n for |v|^2 (q = 1) or 2n(q+1)/2 per point for the batch V^T V."""
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


def cpu_baseline(wl, sample: int):
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = 1
    t0 = time.perf_counter()
    model = O.fit(wl.X, wl.Y, wl.lengthscale, wl.outputscale, wl.noise)
    t1 = time.perf_counter()
    cand = wl.cand[:sample].astype(np.float64)
    out = O.score(model, cand, wl.ref, wl.Z.astype(np.float64))
    O.argmax(out["ehvi"])
    t2 = time.perf_counter()
    return {
        "value": sample / (t2 - t1),
        "unit": "candidates/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"first {sample} candidates of the same workload; fp64 oracle "
                  f"score + argmax took {t2 - t1:.2f} s (fit {t1 - t0:.2f} s, excluded)",
    }


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-sample", type=int, default=65536)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-peaks", action="store_true", help="skip the achieved-peak probes")
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="also run one plain device copy of this many MiB (counter calibration)")
    a = ap.parse_args(argv)

    if a.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        return 2

    import torch
    import bo_inputs as bi
    import paper_2602_10729_amd as bo

    wl = bi.make_config(a.config, seed=a.seed)
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

    def step():
        model = bo.fit(X, Y, wl.lengthscale, wl.outputscale, wl.noise, stream=stream)
        bo.score(model, cand, wl.ref, Z, ehvi=ehvi, stream=stream)
        bo.argmax(ehvi, index=idx, value=val, stream=stream)
        return model

    models = [step() for _ in range(a.warmup)]
    torch.cuda.synchronize()
    del models

    # fit alone (reported, and part of every step)
    t0 = time.perf_counter()
    m0 = bo.fit(X, Y, wl.lengthscale, wl.outputscale, wl.noise, stream=stream)
    fit_ms = (time.perf_counter() - t0) * 1e3
    del m0

    if a.calib_copy_mb > 0:
        nbytes = a.calib_copy_mb << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    bo.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    keep = []
    for _ in range(a.steps):
        keep.append(step())
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    post_ms, ehvi_ms, calls, launches = bo.profile_read()
    bo.profile_enable(False)
    best = int(idx.item())
    del keep

    ms_per_step = (t1 - t0) * 1e3 / a.steps
    value = wl.M / (ms_per_step / 1e3)
    n_pts = wl.M * wl.q
    flops_launch = n_pts * posterior_flops_per_point(wl.n, wl.d, wl.q)
    f16_launch = n_pts * posterior_f16_mfma_flops_per_point(wl.n)
    launch_ms = post_ms / max(launches, 1)
    achieved = f16_launch / (launch_ms / 1e3) / 1e12
    achieved32 = flops_launch / (launch_ms / 1e3) / 1e12
    score_ms = (post_ms + ehvi_ms) / max(calls, 1)

    rec = {
        "metric": METRIC,
        "value": value,
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 (posterior contraction and distance dot products: fp16x3 split products, fp32 accumulate)",
        "data": "synthetic",
        "config": {
            "workload": f"config {a.config}: M={wl.M} candidates (q={wl.q}), n={wl.n} "
                        f"observations, d={wl.d}, m={wl.m} objectives, S={wl.S} MC samples, seed {a.seed}",
            "M": wl.M, "q": wl.q, "n": wl.n, "d": wl.d, "m": wl.m, "S": wl.S,
            "step": "bo_fit + bo_score + bo_argmax",
        },
        "roofline": {
            "bound": "mfma",
            "kernel": "k_posterior (one launch per objective)",
            "mfma_dtype": "f16 (3 split products per multiply-add, fp32 accumulate)",
            "achieved": achieved,
            "peak": PEAK_FP16_MFMA_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_FP16_MFMA_TFLOPS,
            "traffic": recorded_traffic("headline") if a.config == 3 else None,
            "launch_ms": launch_ms,
            "flops_per_launch": f16_launch,
            "fp32_equivalent": {"achieved": achieved32, "peak": PEAK_FP32_MFMA_TFLOPS,
                                "unit": "TFLOP/s", "frac": achieved32 / PEAK_FP32_MFMA_TFLOPS,
                                "flops_per_launch": flops_launch},
        },
        "phases_ms": {"fit": fit_ms, "posterior_per_call": post_ms / max(calls, 1),
                      "ehvi_per_call": ehvi_ms / max(calls, 1), "score_per_call": score_ms},
        "score_only_candidates_per_s": wl.M / (score_ms / 1e3) if score_ms > 0 else None,
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
    models_c = bo.fit(X, Y, wl.lengthscale, wl.outputscale, wl.noise, stream=stream)
    bo.score(models_c, cand, wl.ref, Z, ehvi=ehvi, stream=stream, lower=lower)
    torch.cuda.synchronize()
    bo.profile_enable(True)
    for _ in range(a.steps):
        bo.score(models_c, cand, wl.ref, Z, ehvi=ehvi, stream=stream, lower=lower)
    torch.cuda.synchronize()
    _, cehvi_ms, ccalls, _ = bo.profile_read()
    bo.profile_enable(False)
    del models_c
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
            "achieved": f16_launch / (c_launch / 1e3) / 1e12, "peak": PEAK_FP16_MFMA_TFLOPS,
            "unit": "TFLOP/s", "frac": f16_launch / (c_launch / 1e3) / 1e12 / PEAK_FP16_MFMA_TFLOPS,
            "score_candidates_per_s": wl.M / ((cpost_ms / max(cc, 1) + ehvi_launch_ms) / 1e3),
        }
    # the noisy acquisition (qNEHVI): in-sample draws and per-draw fronts
    # prepared once, then whole-workload scoring calls
    if wl.m in (2, 3):
        ZX = torch.from_numpy(bi.insample_base_samples(wl)).to(dev)
        mn = bo.fit(X, Y, wl.lengthscale, wl.outputscale, wl.noise, stream=stream)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        bo.nehvi_prepare(mn, ZX, wl.ref, stream=stream)
        prep_ms = (time.perf_counter() - t0) * 1e3
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
                       "k_nehvi_ehvi per 262144-point chunk",
            "prepare_ms": prep_ms, "score_ms": nz_ms,
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
    if not a.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(wl, a.cpu_sample)
    print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
