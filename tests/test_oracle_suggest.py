"""Pins of the suggestion-step oracle (Algorithm 1's SUGGEST): properties the
paper fixes for the composed step -- the Sobol fill, invariance to the
objectives' units, the constraints and POF threshold honoured, MOBO picks the
largest EHVI, SOBO picks on the MACE front."""
import numpy as np
import pytest

from oracle.mace import pareto_front_max
from oracle.sobol import known_constraints_mask, sobol_pool
from oracle.suggest import suggest
from tests.suggest_cases import fixed_theta, observations, space

POOL = 512


def _fixed(p, d):
    th = fixed_theta(p, d)
    return dict(theta_lower=th, theta_upper=th)


def test_no_valid_observation_gives_the_first_admissible_sobol_points():
    sp = space()
    pool = sobol_pool(sp["poly"], sp["vinit"], sp["levels"], POOL, 7)
    adm = np.flatnonzero(known_constraints_mask(pool, sp["A"], sp["b"]))
    assert len(adm) < POOL  # the constraint does prune
    for X, Y, v in [(np.zeros((0, 4)), np.zeros((0, 1)), np.zeros(0)),
                    (np.random.default_rng(0).random((5, 4)), np.ones((5, 1)), np.zeros(5))]:
        r = suggest(X, Y, v, sp, k=6, pool_size=POOL, pool_skip=7)
        np.testing.assert_array_equal(r["idx"], adm[:6])
        np.testing.assert_array_equal(r["x"], pool[adm[:6]].astype(np.float64))
        assert np.all(r["source"] == 1)


@pytest.mark.parametrize("p", [1, 2])
def test_units_of_the_objectives_do_not_matter(p):
    """Scaling every objective by a power of two (exact) and shifting it
    changes nothing: the step standardises first, and MLE runs on the same
    numbers."""
    sp = space()
    X, Y, v = observations(24, p=p)
    a = suggest(X, Y, v, sp, k=3, pool_size=POOL, t=4, pick_seed=5, n_trees=8, max_depth=4)
    b = suggest(X, 4.0 * Y, v, sp, k=3, pool_size=POOL, t=4, pick_seed=5, n_trees=8, max_depth=4)
    np.testing.assert_array_equal(a["idx"], b["idx"])
    np.testing.assert_array_equal(a["theta"], b["theta"])


@pytest.mark.parametrize("p", [1, 2])
def test_picks_honour_known_constraints_and_pof(p):
    sp = space()
    X, Y, v = observations(30, p=p)
    assert 0 < v.sum() < len(v)
    r = suggest(X, Y, v, sp, k=4, delta=0.6, pool_size=POOL, n_trees=8, max_depth=4, **_fixed(p, 4))
    solver = r["idx"][r["source"] == 0]
    assert len(solver) == 4
    assert np.all(r["mask"][solver] == 1) and np.all(r["known"][solver] == 1)
    x = r["x"]
    assert np.all(x[:, 0] - x[:, 1] <= 0.3)


def test_mobo_picks_the_largest_ehvi():
    sp = space()
    X, Y, v = observations(30, p=2)
    r = suggest(X, Y, v, sp, k=4, pool_size=POOL, n_trees=8, max_depth=4, **_fixed(2, 4))
    acq, mask, idx = r["acq"], r["mask"], r["idx"]
    rest = np.setdiff1d(np.flatnonzero(mask), idx)
    assert np.all(np.diff(acq[idx]) <= 0)  # in order
    assert acq[idx].min() >= acq[rest].max()


def test_sobo_picks_lie_on_the_mace_front():
    sp = space()
    X, Y, v = observations(30, p=1)
    r = suggest(X, Y, v, sp, k=4, pool_size=POOL, n_trees=8, max_depth=4, t=3, pick_seed=9, **_fixed(1, 4))
    S = np.stack([r["ucb"], r["pi"], r["ei"]], axis=1)
    elig = np.flatnonzero(r["mask"])
    for i in r["idx"]:
        dom = np.all(S[elig] >= S[i], axis=1) & np.any(S[elig] > S[i], axis=1)
        assert not dom.any()
    assert np.array_equal(r["front"], pareto_front_max(S, r["mask"]))


def test_shortfall_is_filled_in_sobol_order():
    """Delta = 1 admits only candidates every tree calls feasible; the rest of
    the k come from the pool in order, admissible and not already picked."""
    sp = space()
    X, Y, v = observations(30, p=2)
    r = suggest(X, Y, v, sp, k=8, delta=1.0, pool_size=64, n_trees=8, max_depth=4, **_fixed(2, 4))
    src, idx = r["source"], r["idx"]
    n_solver = int((src == 0).sum())
    assert n_solver == min(8, int(r["mask"].sum()))
    fill = idx[n_solver:]
    adm = [i for i in np.flatnonzero(r["known"]) if i not in set(idx[:n_solver])]
    np.testing.assert_array_equal(fill, adm[:len(fill)])
    assert len(idx) == 8


def test_fixed_hyperparameters_are_used_as_given():
    sp = space()
    X, Y, v = observations(20, p=2)
    r = suggest(X, Y, v, sp, k=2, pool_size=64, n_trees=4, max_depth=3, **_fixed(2, 4))
    np.testing.assert_array_equal(r["theta"], fixed_theta(2, 4))


def test_learned_warp_is_at_least_as_likely_as_the_identity():
    """With the warping learned (the paper's covariance), every objective's
    likelihood at the learned parameters is at least that of the search
    without warping, the warp parameters stay in their box, and the
    suggestion is still a set of distinct admissible pool points."""
    from oracle.mle import nll_and_grad, nll_and_grad_warp
    from oracle.suggest import WARP_LOWER, WARP_UPPER
    sp = space()
    X, Y, v = observations(30, p=2)
    rw = suggest(X, Y, v, sp, k=3, pool_size=POOL, kernel="matern32", learn_warp=True)
    r0 = suggest(X, Y, v, sp, k=3, pool_size=POOL, kernel="matern32")
    d = len(sp["levels"])
    ok = v != 0
    Yv = Y[ok]
    Ys = (Yv - Yv.mean(axis=0)) / np.where(Yv.std(axis=0) > 0, Yv.std(axis=0), 1.0)
    assert rw["theta"].shape == (2, 3 * d + 2)
    for j in range(2):
        fw, _ = nll_and_grad_warp(rw["theta"][j], X[ok], Ys[:, j], "matern32")
        f0, _ = nll_and_grad(r0["theta"][j], X[ok], Ys[:, j], "matern32")
        assert fw <= f0 + 1e-9
        w = np.exp(rw["theta"][j][d + 2:])
        assert np.all(w >= WARP_LOWER * (1 - 1e-12)) and np.all(w <= WARP_UPPER * (1 + 1e-12))
    assert len(set(rw["idx"].tolist())) == len(rw["idx"]) == 3
