"""Hypervolume, hypervolume improvement and EHVI: Sec. 4.4.2, Eq. 9, Fig. 4.

All objectives are minimised, so the reference point r is an UPPER bound and
the region a set S dominates is the union of the boxes [s, r] over s in S.
(The paper maximises and takes r as a lower bound; the mirror is exact.)

HV_r(S)   = volume( union_{s in S} [s, r] )
HVI(y; S) = HV_r(S + {y}) - HV_r(S)                     (never negative)
EHVI(x)   = E[ HVI(Y; P) ],  Y_j ~ N(mu_j(x), sigma_j(x)^2) independent (Eq. 9)

Closed form used here.  Let A be the part of the region below r that no point
of the front P dominates.  The sorted coordinates of P and r, with -inf
prepended, cut space into a grid; each grid cell lies wholly inside A or wholly
outside it, and a cell [l, u] is inside A iff no p in P satisfies p <= l.
For any y, [y, r] intersected with A is the part of the new box not yet
covered, so HVI(y) = sum over cells B in A of prod_j (u_Bj - max(l_Bj, y_j))^+.
Each factor equals (u - y)^+ - (l - y)^+, and the objectives are independent
(Sec. 4.3), hence

    EHVI = sum_B prod_j ( G_j(u_Bj) - G_j(l_Bj) ),   G_j(c) = E[(c - Y_j)^+],

with G_j(-inf) = 0 (``acquisition.partial_expectation``).
"""
import itertools

import numpy as np

from .acquisition import partial_expectation


def nondominated(Y, ref):
    """The front of Y with respect to r: rows strictly below r in every
    coordinate that no other row weakly dominates; duplicates kept once.
    Returned sorted lexicographically."""
    Y = np.asarray(Y, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    cand = np.unique(Y[np.all(Y < ref, axis=1)], axis=0)
    keep = []
    for i, p in enumerate(cand):
        dominated = False
        for j, q in enumerate(cand):
            if j != i and np.all(q <= p) and np.any(q < p):
                dominated = True
                break
        if not dominated:
            keep.append(p)
    if not keep:
        return np.zeros((0, Y.shape[1]))
    return np.array(sorted(map(tuple, keep)))


def _axes(P, ref):
    """Grid coordinates per objective: -inf, the front's sorted values, r."""
    return [np.concatenate(([-np.inf], np.unique(P[:, j]), [ref[j]])) for j in range(len(ref))]


def hypervolume(S, ref):
    """HV_r(S) by summing the grid cells that some point of S dominates."""
    S = np.asarray(S, dtype=np.float64).reshape(-1, len(ref))
    ref = np.asarray(ref, dtype=np.float64)
    S = S[np.all(S < ref, axis=1)]
    if len(S) == 0:
        return 0.0
    axes = [np.concatenate((np.unique(S[:, j]), [ref[j]])) for j in range(len(ref))]
    total = 0.0
    for idx in itertools.product(*[range(len(a) - 1) for a in axes]):
        lo = np.array([axes[j][i] for j, i in enumerate(idx)])
        hi = np.array([axes[j][i + 1] for j, i in enumerate(idx)])
        if np.any(np.all(S <= lo, axis=1)):
            total += float(np.prod(hi - lo))
    return total


def hypervolume_2d_rectangles(S, ref):
    """Two objectives: the sum of the rectangles each front point adds when the
    front is walked in order of the first objective (the construction drawn in
    Fig. 4a)."""
    P = nondominated(S, ref)
    total = 0.0
    prev_y2 = ref[1]
    for p in P[np.argsort(P[:, 0])]:
        total += (ref[0] - p[0]) * (prev_y2 - p[1])
        prev_y2 = p[1]
    return total


def hypervolume_improvement(y, S, ref):
    """HVI(y; S) = HV(S + {y}) - HV(S), for a single point y."""
    S = np.asarray(S, dtype=np.float64).reshape(-1, len(ref))
    return hypervolume(np.vstack([S, np.asarray(y, dtype=np.float64)[None, :]]), ref) - hypervolume(S, ref)


def nondominated_cells(P, ref):
    """Every grid cell of the region A below r that the front P leaves open.

    Returns (lo, hi), each (n_cells, p); lo may hold -inf."""
    P = np.asarray(P, dtype=np.float64).reshape(-1, len(ref))
    axes = _axes(P, ref)
    lo_list, hi_list = [], []
    for idx in itertools.product(*[range(len(a) - 1) for a in axes]):
        lo = np.array([axes[j][i] for j, i in enumerate(idx)])
        hi = np.array([axes[j][i + 1] for j, i in enumerate(idx)])
        if len(P) and np.any(np.all(P <= lo, axis=1)):
            continue
        lo_list.append(lo)
        hi_list.append(hi)
    return np.array(lo_list), np.array(hi_list)


def column_boxes(P, ref):
    """The same open region A, with the cells of each column along the last
    objective merged: over each cell of the first p-1 coordinates the open part
    is [-inf, h] in the last one, h = min of r and of the last coordinate of the
    front points dominating the column's lower corner."""
    P = np.asarray(P, dtype=np.float64).reshape(-1, len(ref))
    ref = np.asarray(ref, dtype=np.float64)
    p = len(ref)
    axes = _axes(P, ref)[:-1]
    lo_list, hi_list = [], []
    for idx in itertools.product(*[range(len(a) - 1) for a in axes]):
        lo = np.array([axes[j][i] for j, i in enumerate(idx)])
        hi = np.array([axes[j][i + 1] for j, i in enumerate(idx)])
        h = ref[p - 1]
        if len(P):
            dom = np.all(P[:, :p - 1] <= lo, axis=1)
            if np.any(dom):
                h = min(h, float(np.min(P[dom, p - 1])))
        lo_list.append(np.concatenate((lo, [-np.inf])))
        hi_list.append(np.concatenate((hi, [h])))
    return np.array(lo_list), np.array(hi_list)


def hvi_from_boxes(y, lo, hi):
    """HVI(y) = sum_B prod_j (u_Bj - max(l_Bj, y_j))^+ for one point y."""
    y = np.asarray(y, dtype=np.float64)
    return float(np.sum(np.prod(np.maximum(hi - np.maximum(lo, y), 0.0), axis=1)))


def ehvi(mu, sigma, P, ref, boxes="columns", chunk=4096):
    """EHVI for every candidate (Eq. 9).  mu, sigma: (n, p) arrays."""
    mu = np.atleast_2d(np.asarray(mu, dtype=np.float64))
    sigma = np.atleast_2d(np.asarray(sigma, dtype=np.float64))
    lo, hi = (column_boxes if boxes == "columns" else nondominated_cells)(P, ref)
    n = mu.shape[0]
    out = np.zeros(n)
    for s in range(0, n, chunk):
        m = mu[s:s + chunk]
        sd = sigma[s:s + chunk]
        acc = np.zeros(len(m))
        for b in range(len(lo)):
            term = np.ones(len(m))
            for j in range(mu.shape[1]):
                gu = partial_expectation(hi[b, j], m[:, j], sd[:, j])
                gl = partial_expectation(lo[b, j], m[:, j], sd[:, j])
                term *= gu - gl
            acc += term
        out[s:s + chunk] = acc
    return out


def reference_point(Y, margin=0.1):
    """r_j = worst observed + margin * observed range, per objective."""
    Y = np.asarray(Y, dtype=np.float64)
    mx, mn = Y.max(axis=0), Y.min(axis=0)
    return mx + margin * (mx - mn)
