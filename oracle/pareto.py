"""Pareto front and box decompositions, fp64 (test infrastructure only).

The paper's acquisition (constrained qNEHVI paragraph) is built on the
hypervolume improvement over the current Pareto front of the observed
objective vectors; neither the front nor a decomposition is spelled out
there. Readings used:

* Maximisation. y_j dominates y_i when y_j >= y_i componentwise and
  y_j != y_i. Exact duplicates keep the lowest index. Only points strictly
  above the reference point r in every objective are kept. The front is
  sorted by objective 0 ascending (ties by index).
* The region a new point can improve is {z > r : no f in F with f >= z}.
  It is covered by disjoint axis-aligned boxes [lo, hi) (hi may be +inf):
  - m = 2: the staircase below the front, P + 1 boxes;
  - m = 3: a sweep along objective 2 from the top: between consecutive
    objective-2 levels of the front the active points (those at or above the
    level) cast a 2-D staircase; staircase boxes that persist from one level
    to the next are merged into one taller box.
"""
from __future__ import annotations

import numpy as np


def nondominated(Y: np.ndarray) -> np.ndarray:
    """Indices of non-dominated rows of Y (maximise), duplicates dropped.

    Brute force over all pairs (one n x n comparison per objective);
    returned in increasing index order. Row i is dropped when some row j is
    >= it in every objective and differs in one, or equals it with j < i.
    """
    Y = np.asarray(Y, dtype=np.float64)
    n = Y.shape[0]
    ge = np.ones((n, n), dtype=bool)        # ge[i, j]: Y[j] >= Y[i] componentwise
    ne = np.zeros((n, n), dtype=bool)       # ne[i, j]: Y[j] != Y[i] somewhere
    for k in range(Y.shape[1]):
        col = Y[:, k]
        ge &= col[None, :] >= col[:, None]
        ne |= col[None, :] != col[:, None]
    dominated = np.any(ge & ne, axis=1)
    earlier_dup = np.any(np.tril(~ne, -1), axis=1)     # an equal row j < i
    return np.nonzero(~(dominated | earlier_dup))[0]


def pareto_front(Y: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Front indices: non-dominated, strictly above ref, sorted by obj 0."""
    Y = np.asarray(Y, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    idx = nondominated(Y)
    idx = idx[np.all(Y[idx] > ref, axis=1)]
    order = np.argsort(Y[idx, 0], kind="stable")
    return idx[order]


def _staircase(P2: np.ndarray, r0: float, r1: float):
    """2-D boxes (xlo, xhi, ylo) covering the part of (r0,inf)x(r1,inf) not
    weakly dominated by any point of P2 (upper y bound is +inf)."""
    if len(P2) == 0:
        return [(r0, np.inf, r1)]
    # scan by x descending (ties: y descending); a point is 2-D non-dominated
    # when its y beats every point with larger or equal x seen so far
    order = np.lexsort((-P2[:, 1], -P2[:, 0]))
    nd = []
    best_y = -np.inf
    for x, y in P2[order]:
        if y > best_y:
            nd.append((x, y))
            best_y = y
    nd = nd[::-1]                    # x ascending, y descending
    boxes = []
    xlo = r0
    for x, y in nd:
        if x > xlo:
            boxes.append((xlo, x, y))
        xlo = max(xlo, x)
    boxes.append((xlo, np.inf, r1))
    return boxes


def boxes_2d(F: np.ndarray, ref: np.ndarray):
    """Staircase boxes for m = 2: lo [P+1, 2], hi [P+1, 2].

    With F sorted by objective 0 ascending: box i spans objective 0 from
    l_i to u_i (l_1 = r_0, l_{i+1} = u_i = f_i,0, u_{P+1} = inf) and
    objective 1 from h_i (= f_i,1, h_{P+1} = r_1) to inf.
    """
    F = np.asarray(F, dtype=np.float64).reshape(-1, 2)
    ref = np.asarray(ref, dtype=np.float64)
    P = F.shape[0]
    lo = np.empty((P + 1, 2))
    hi = np.empty((P + 1, 2))
    xs = np.concatenate([[ref[0]], F[:, 0]])
    lo[:, 0] = xs
    hi[:P, 0] = F[:, 0]
    hi[P, 0] = np.inf
    lo[:P, 1] = F[:, 1]
    lo[P, 1] = ref[1]
    hi[:, 1] = np.inf
    return lo, hi


def boxes_3d(F: np.ndarray, ref: np.ndarray):
    """Disjoint boxes for m = 3 by a sweep along objective 2 (see module doc)."""
    F = np.asarray(F, dtype=np.float64).reshape(-1, 3)
    ref = np.asarray(ref, dtype=np.float64)
    order = np.argsort(-F[:, 2], kind="stable")
    open_boxes = {b: np.inf for b in _staircase(F[:0, :2], ref[0], ref[1])}
    out = []
    active = []
    for j in order:
        zb = F[j, 2]
        active.append(F[j, :2])
        new = set(_staircase(np.array(active), ref[0], ref[1]))
        for key in list(open_boxes):
            if key not in new:
                ztop = open_boxes.pop(key)
                if ztop > zb:
                    out.append((key[0], key[2], zb, key[1], np.inf, ztop))
        for key in new:
            if key not in open_boxes:
                open_boxes[key] = zb
    for key, ztop in open_boxes.items():
        if ztop > ref[2]:
            out.append((key[0], key[2], ref[2], key[1], np.inf, ztop))
    arr = np.array(out, dtype=np.float64).reshape(-1, 6)
    return arr[:, :3].copy(), arr[:, 3:].copy()


def box_decomposition(F: np.ndarray, ref: np.ndarray):
    """Dispatch on the number of objectives (2 or 3)."""
    m = np.asarray(ref).shape[0]
    if m == 2:
        return boxes_2d(F, ref)
    if m == 3:
        return boxes_3d(F, ref)
    raise ValueError("box decomposition implemented for m in {2, 3}")
