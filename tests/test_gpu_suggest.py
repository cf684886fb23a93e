"""The suggestion step end to end (scoot_suggest: Algorithm 1's SUGGEST)
against the oracle's, and Algorithm 1 driven by a synthetic evaluator.

With the hyperparameters fixed the two sides see identical inputs: the pool,
the known mask and the forest votes are bit-exact, so the configurations must
match exactly in float64 -- except where the oracle's own ranking has a near
tie at the cut (two candidates whose scores differ by less than the float
bar), where any of the tied candidates is right.  The Sobol fill is exact."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2408_04323_amd as S  # noqa: E402
from oracle.mle import fit_hyperparameters, nll_and_grad  # noqa: E402
from oracle.suggest import suggest as oracle_suggest  # noqa: E402
from oracle.threshold import delta_update  # noqa: E402
from tests.suggest_cases import evaluate, fixed_theta, observations, space  # noqa: E402

pytestmark = pytest.mark.gpu


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def _rows(x):
    return [tuple(r) for r in np.asarray(x, dtype=np.float64)]


def check_against_oracle(got_x, got_src, want, k, p, dtype):
    """got_x / got_src from the library; want the oracle's dict."""
    assert len(got_x) == len(want["x"])
    np.testing.assert_array_equal(got_src, want["source"])
    pool = want["pool"].astype(np.float64)
    index = {r: i for i, r in reversed(list(enumerate(_rows(pool))))}
    got_idx = np.array([index[r] for r in _rows(got_x)])
    n_solver = int((want["source"] == 0).sum())
    # the fill is exact
    np.testing.assert_array_equal(got_idx[n_solver:], want["idx"][n_solver:])
    if n_solver == 0 or np.array_equal(got_idx, want["idx"]):
        return
    # solver picks differ: only allowed at a near tie of the oracle's ranking
    assert p > 1, "one objective: the MACE pick must match exactly in float64"
    acq, mask = want["acq"], want["mask"]
    tol = (1e-3 if dtype == "f32" else 1e-10) * acq.max()
    assert np.all(mask[got_idx[:n_solver]] == 1)
    kth = acq[want["idx"][n_solver - 1]]
    assert np.all(acq[got_idx[:n_solver]] >= kth - 2 * tol), "a pick below the oracle's k-th best"
    elig = np.sort(acq[mask == 1])[::-1]
    gap = elig[n_solver - 1] - (elig[n_solver] if len(elig) > n_solver else -np.inf)
    assert gap <= 2 * tol, "picks differ although the oracle's cut is clear"


CASES = [  # (p, dtype, n_obs, delta, k)
    (1, "f64", 24, 0.5, 4),
    (2, "f64", 30, 0.5, 4),
    (2, "f32", 30, 0.6, 3),
    (3, "f64", 36, 0.5, 2),
    (2, "f64", 30, 1.0, 8),   # shortfall: Delta = 1
]


@pytest.mark.parametrize("p,dtype,n_obs,delta,k", CASES)
def test_suggest_matches_oracle(p, dtype, n_obs, delta, k):
    sp = space()
    X, Y, v = observations(n_obs, p=p, seed=7 + p)
    th = fixed_theta(p, 4)
    kw = dict(k=k, delta=delta, pool_size=2048 + 5, pool_skip=3, theta_lower=th, theta_upper=th, n_trees=8,
              max_depth=5, forest_seed=17, t=5, pick_seed=99)
    say("suggest", p, dtype, n_obs, delta, k)
    x, src, theta = S.suggest(X, Y, v, sp, dtype=dtype, **kw)
    want = oracle_suggest(X, Y, v, sp, **kw)
    np.testing.assert_array_equal(theta, th)
    check_against_oracle(x, src, want, k, p, dtype)
    assert np.all(x[:, 0] - x[:, 1] <= 0.3)


def test_suggest_without_valid_observations_is_the_sobol_fill():
    sp = space()
    for n_obs in (0, 6):
        X = np.random.default_rng(1).random((n_obs, 4))
        say("suggest fill", n_obs)
        x, src, theta = S.suggest(X, np.ones((n_obs, 2)), np.zeros(n_obs), sp, k=5, pool_size=300, pool_skip=11)
        want = oracle_suggest(X, np.ones((n_obs, 2)), np.zeros(n_obs), sp, k=5, pool_size=300, pool_skip=11)
        np.testing.assert_array_equal(x, want["x"])
        assert np.all(src == 1) and np.all(np.isnan(theta))


def test_suggest_learns_hyperparameters():
    """With the search on, the step's hyperparameters are a likelihood optimum
    at least as good as the oracle's from the same start, and the rest of the
    step is the fixed-hyperparameter step at that optimum."""
    sp = space()
    X, Y, v = observations(28, p=2, seed=21)
    kw = dict(k=3, pool_size=1024, n_trees=8, max_depth=5, forest_seed=4)
    say("suggest with mle")
    x, src, theta = S.suggest(X, Y, v, sp, **kw)
    ok = v != 0
    Ys = (Y[ok] - Y[ok].mean(0)) / Y[ok].std(0)
    lo = np.log(np.array([0.01] * 4 + [0.05, 1e-6]))
    hi = np.log(np.array([10.0] * 4 + [20.0, 1.0]))
    start = np.log(np.array([0.5] * 4 + [1.0, 1e-3]))
    for j in range(2):
        _, f_o = fit_hyperparameters(X[ok], Ys[:, j], start, lo, hi)
        f_g, _ = nll_and_grad(theta[j], X[ok], Ys[:, j])
        assert f_g <= f_o + 1e-6 * max(1.0, abs(f_o))
        assert np.all(theta[j] >= lo) and np.all(theta[j] <= hi)
    x2, src2, _ = S.suggest(X, Y, v, sp, theta_lower=theta, theta_upper=theta, **kw)
    np.testing.assert_array_equal(x2, x)
    np.testing.assert_array_equal(src2, src)


@pytest.mark.parametrize("p", [1, 2])
def test_algorithm1_loop(p):
    """Algorithm 1 with a synthetic evaluator that crashes in part of the
    space: the initial Sobol design (as many points as dimensions), then
    rounds of SUGGEST(k), EVALUATE, the Delta update and the union of the
    observations.  The oracle drives the sequence; at every round the
    library's suggestion from the same observations is checked against it, and
    the library's Delta update against the oracle's."""
    sp = space()
    d, k, N = 4, 2, 16
    th = fixed_theta(p, d)
    kw = dict(pool_size=1024, theta_lower=th, theta_upper=th, n_trees=8, max_depth=5)
    X = np.zeros((0, d))
    Y = np.zeros((0, p))
    v = np.zeros(0, np.uint8)
    want = oracle_suggest(X, Y, v, sp, k=d, **kw)
    x, _, _ = S.suggest(X, Y, v, sp, k=d, dtype="f64", **kw)
    np.testing.assert_array_equal(x, want["x"])
    y_new, v_new = evaluate(want["x"], p)
    X, Y, v = want["x"], y_new, v_new
    delta, c = 0.5, 0
    rnd = 1
    while len(X) < N:
        say("algorithm 1 round", p, rnd, len(X), delta)
        args = dict(k=k, delta=delta, pool_skip=1024 * rnd, t=rnd, pick_seed=rnd, forest_seed=rnd, **kw)
        want = oracle_suggest(X, Y, v, sp, **args)
        x, src, _ = S.suggest(X, Y, v, sp, dtype="f64", **args)
        check_against_oracle(x, src, want, k, p, "f64")
        y_new, v_new = evaluate(want["x"], p)
        any_invalid = bool((v_new == 0).any())
        d_lib, c_lib = S.delta_update(delta, c, k, any_invalid)
        delta, c = delta_update(delta, c, k, any_invalid)
        assert (d_lib, c_lib) == (delta, c)
        X, Y, v = np.vstack([X, want["x"]]), np.vstack([Y, y_new]), np.concatenate([v, v_new])
        rnd += 1
    assert 0.25 <= delta <= 0.75


def test_suggest_learns_the_warping():
    """With learn_warp (the paper's Matern-3/2 with input warping learned with
    the GP), each objective's parameters (3d + 2: lengthscales, variances and
    the Kumaraswamy a, b) are a likelihood optimum at least as good as the
    oracle's from the same start and inside their boxes, and the rest of the
    step is the fixed-parameter step at that optimum (the same picks with the
    learned warp and hyperparameters given)."""
    from oracle.mle import fit_hyperparameters_warp, nll_and_grad_warp
    sp = space()
    X, Y, v = observations(28, p=2, seed=23)
    d = 4
    kw = dict(k=3, pool_size=1024, n_trees=8, max_depth=5, forest_seed=4, kernel="matern32")
    say("suggest learning the warp")
    x, src, theta = S.suggest(X, Y, v, sp, learn_warp=True, **kw)
    assert theta.shape == (2, 3 * d + 2)
    ok = v != 0
    Ys = (Y[ok] - Y[ok].mean(0)) / Y[ok].std(0)
    lo = np.log(np.array([0.01] * d + [0.05, 1e-6] + [0.2] * (2 * d)))
    hi = np.log(np.array([10.0] * d + [20.0, 1.0] + [5.0] * (2 * d)))
    start = np.log(np.array([0.5] * d + [1.0, 1e-3] + [1.0] * (2 * d)))
    for j in range(2):
        _, f_o = fit_hyperparameters_warp(X[ok], Ys[:, j], start, lo, hi, "matern32")
        f_g, _ = nll_and_grad_warp(theta[j], X[ok], Ys[:, j], "matern32")
        assert f_g <= f_o + 1e-6 * max(1.0, abs(f_o))
        assert np.all(theta[j] >= lo - 1e-12) and np.all(theta[j] <= hi + 1e-12)
    th = theta[:, :d + 2]
    x2, src2, _ = S.suggest(X, Y, v, sp, theta_lower=th, theta_upper=th, warp_a=np.exp(theta[:, d + 2:2 * d + 2]),
                            warp_b=np.exp(theta[:, 2 * d + 2:]), **kw)
    np.testing.assert_array_equal(x2, x)
    np.testing.assert_array_equal(src2, src)
