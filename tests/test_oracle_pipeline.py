"""Pins of the oracle's whole scoring pass (Sec. 4.1, steps 3-8: posterior per
objective, acquisition, feasibility mask, top-q) on hand-worked workloads.

With a single observation every quantity has a closed form (Eq. 4-5 with
m = 1): k(x) the covariance to the observation,

    mu(x)      = c + k(x) (y - c) / (s^2 + tau^2),
    sigma^2(x) = s^2 - k(x)^2 / (s^2 + tau^2).

EI (Eq. 8, minimised) and the 2-D EHVI (Eq. 9) over a front of at most one
point are then written out here from scipy's normal distribution, and the
feasibility votes of two hand-built stumps are counted by hand, so the pick is
known in advance: with y above the prior mean a farther candidate has both a
lower mean and a larger deviation, hence a larger EI, so the pick is the
farthest feasible candidate (the farthest candidate of all is infeasible).
"""
import math

import numpy as np
import pytest
from scipy.stats import norm

from oracle.pipeline import score_pool

# candidates: index 0 is the farthest but infeasible (no vote), 1 is the
# farthest feasible with exactly half of the votes (POF = Delta, inclusive),
# 2 the next, 3 and 5 near the observation, 4 far but infeasible.
XC = np.array([[0.05, 0.95], [0.93, 0.95], [0.10, 0.10], [0.50, 0.55], [0.15, 0.92], [0.60, 0.20]])
X_OBS = np.array([[0.5, 0.5]])
# two stumps: tree 0 votes 1 when x0 > 0.2, tree 1 votes 1 when x1 <= 0.9
STUMPS = dict(feature=np.array([0, 0, 0, 1, 0, 0], np.int32),
              threshold=np.array([0.2, 0, 0, 0.9, 0, 0], np.float32),
              left=np.array([1, -1, -1, 1, -1, -1], np.int32), right=np.array([2, -1, -1, 2, -1, -1], np.int32),
              leaf_q16=np.array([0, 0, 65536, 0, 65536, 0], np.int32), tree_offset=np.array([0, 3, 6], np.int64))
VOTES = np.array([0, 65536, 65536, 131072, 0, 131072])


def _matern52(x, X, ls, s2):
    r = math.sqrt(sum(((a - b) / l) ** 2 for a, b, l in zip(x, X, ls)))
    return s2 * (1 + math.sqrt(5) * r + 5 * r * r / 3) * math.exp(-math.sqrt(5) * r)


def _closed_form(y, c, ls, s2, tau2):
    k = np.array([_matern52(x, X_OBS[0], ls, s2) for x in XC])
    mu = c + k * (y - c) / (s2 + tau2)
    sd = np.sqrt(s2 - k * k / (s2 + tau2))
    return mu, sd


def _G(cut, mu, sd):
    """E[(cut - Y)^+] for Y ~ N(mu, sd^2), from scipy's normal distribution."""
    u = (cut - mu) / sd
    return sd * (u * norm.cdf(u) + norm.pdf(u))


def _workload(p, Y, lengthscale, signal_var, noise_var, prior_mean, ref=None, q=2, delta=0.5):
    return dict(X=X_OBS, Y=np.asarray(Y, float).reshape(1, p), lengthscale=np.asarray(lengthscale, float),
                signal_var=np.asarray(signal_var, float), noise_var=np.asarray(noise_var, float),
                prior_mean=np.asarray(prior_mean, float), best_y=float(np.asarray(Y).ravel()[0]), xi=1e-4,
                ref=None if ref is None else np.asarray(ref, float), forest=STUMPS, delta=delta, q=q, Xc=XC)


def test_single_objective_pass_by_hand():
    w = _workload(1, [0.3], [[0.2, 0.4]], [1.0], [0.01], [0.0])
    r = score_pool(w)
    mu, sd = _closed_form(0.3, 0.0, [0.2, 0.4], 1.0, 0.01)
    np.testing.assert_allclose(r["mu"][:, 0], mu, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(r["sigma"][:, 0], sd, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(r["acq"], _G(0.3 + 1e-4, mu, sd), rtol=1e-12, atol=1e-15)
    np.testing.assert_array_equal(r["votes"], VOTES)
    np.testing.assert_array_equal(r["mask"], [0, 1, 1, 1, 0, 1])
    # EI grows with the distance to the observation: the farthest feasible first
    assert np.argmax(r["acq"]) == 0
    np.testing.assert_array_equal(r["idx"], [1, 2])
    assert r["n_valid"] == 4


def test_single_objective_pick_moves_with_delta():
    """Delta = 0.75 needs both votes (threshold ceil(0.75 * 2 * 65536) = 98304):
    only candidates 3 and 5 stay, and 5 is the farther."""
    w = _workload(1, [0.3], [[0.2, 0.4]], [1.0], [0.01], [0.0], delta=0.75)
    r = score_pool(w)
    np.testing.assert_array_equal(r["mask"], [0, 0, 0, 1, 0, 1])
    np.testing.assert_array_equal(r["idx"], [5, 3])
    assert r["n_valid"] == 2


@pytest.mark.parametrize("ref,front_size", [([1.0, 1.0], 1), ([0.25, 1.0], 0)])
def test_two_objective_pass_by_hand(ref, front_size):
    """Objectives with their own lengthscales, variances, noise and prior means.
    The front is the observation when it lies below the reference point, else
    empty.  The non-dominated region of a one-point front p splits into the
    strips (-inf, p0] x (-inf, r1] and [p0, r0] x (-inf, p1], so

        EHVI = G0(p0) G1(r1) + (G0(r0) - G0(p0)) G1(p1),

    and with an empty front it is the single box: G0(r0) G1(r1)."""
    Y = [0.3, -0.2]
    ls = [[0.2, 0.4], [0.5, 0.1]]
    s2, tau2, c = [1.0, 2.0], [0.01, 0.04], [0.0, 0.1]
    w = _workload(2, Y, ls, s2, tau2, c, ref=ref, q=3)
    r = score_pool(w)
    mu = np.empty((6, 2))
    sd = np.empty((6, 2))
    for j in range(2):
        mu[:, j], sd[:, j] = _closed_form(Y[j], c[j], ls[j], s2[j], tau2[j])
    np.testing.assert_allclose(r["mu"], mu, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(r["sigma"], sd, rtol=1e-13, atol=1e-15)
    G = [lambda t, j=j: _G(t, mu[:, j], sd[:, j]) for j in range(2)]
    if front_size:
        want = G[0](Y[0]) * G[1](ref[1]) + (G[0](ref[0]) - G[0](Y[0])) * G[1](Y[1])
    else:
        want = G[0](ref[0]) * G[1](ref[1])
    assert len(r["front"]) == front_size
    np.testing.assert_allclose(r["acq"], want, rtol=1e-12, atol=1e-15)
    elig = np.flatnonzero(VOTES >= 65536)
    order = elig[np.argsort(-want[elig], kind="stable")]
    np.testing.assert_array_equal(r["idx"], order[:3])
    assert r["n_valid"] == 4
