"""fp64 CPU oracle for batch acquisition scoring (test infrastructure only).

This package is the correctness reference that the GPU library is checked
against. It is NOT part of the product path: only the test-suite, the smoke
check and the benchmark's CPU-baseline leg import it. It shares no code,
tables or constants with the GPU library; the only thing the two sides have
in common is the seeded input generator in ``bo_inputs``.

What it computes, step by step (paper: Section "Online Optimization Phase" —
the surrogate-fitting and acquisition-optimisation steps of the MOBO
workflow, the constrained qNEHVI paragraph, and the implementation section
"MOBO optimization kernels"):

* ``gp``      — ARD Matern-5/2 covariance with an output scale (and the
                paper's composite kernel), exact GP conditioning by
                Cholesky, posterior mean / variance / q-batch covariance and
                its PSD Cholesky factor, and the exact log marginal
                likelihood with its gradient.
* ``pareto``  — non-dominated set of the observations and a disjoint box
                decomposition of the region a new point can improve.
* ``acq``     — hypervolume improvement of one point or of a q-batch
                (inclusion-exclusion), Monte-Carlo EHVI / qEHVI with given
                base samples, optionally weighted by the feasibility
                indicator of the constrained form, and the argmax over
                candidates.
* ``noisy``   — the noisy form (qNEHVI): joint posterior samples of
                the latent objectives at the observed points and the
                candidate (or q-batch), a Pareto front per sample of the in-sample values,
                and the candidate's HVI against it, optionally constrained.

All arithmetic is fp64 on fp32-rounded inputs. Readings of points the paper
leaves open are listed in each function's docstring.
"""
from .gp import (GPModel, Composite, matern52, matern32, composite_cov, pref_weight,
                 scaled_distance, fit, posterior, mll,
                 chol_psd, NotPositiveDefinite)
from .pareto import nondominated, pareto_front, boxes_2d, boxes_3d, box_decomposition
from .acq import hvi, qhvi, feasible, ehvi_q1, qehvi, score, argmax
from .noisy import (insample_posterior, insample_samples, candidate_samples, batch_samples,
                    sample_boxes, nehvi)

__all__ = [
    "GPModel", "Composite", "matern52", "matern32", "composite_cov", "pref_weight",
    "scaled_distance", "fit", "posterior", "mll", "chol_psd",
    "NotPositiveDefinite", "nondominated", "pareto_front", "boxes_2d",
    "boxes_3d", "box_decomposition", "hvi", "qhvi", "feasible", "ehvi_q1", "qehvi",
    "score", "argmax", "insample_posterior", "insample_samples", "candidate_samples",
    "batch_samples", "sample_boxes", "nehvi",
]
