"""Pins of the Kriging-believer oracle (sequential extension of Sec. 4.6)."""
import numpy as np
import pytest

from oracle.believer import kriging_believer
from oracle.gp import gp_fit, gp_posterior, matern52
from oracle.hypervolume import ehvi, nondominated
from oracle.pipeline import score_pool
from workloads import make_workload


def test_believer_keeps_mean_and_downdates_variance():
    rng = np.random.default_rng(31)
    X = rng.random((20, 3))
    y = np.cos(4 * X).sum(axis=1)
    ls, s2, t2 = [0.4, 0.6, 0.5], 1.0, 1e-3
    f = gp_fit(X, y, ls, s2, t2)
    Xc = rng.random((200, 3))
    mu, sd = gp_posterior(f, Xc)
    i = 17
    f2 = gp_fit(np.vstack([X, Xc[i:i + 1]]), np.append(y, mu[i]), ls, s2, t2)
    mu2, sd2 = gp_posterior(f2, Xc)
    # the fantasy equals the prediction, so the mean does not move
    np.testing.assert_allclose(mu2, mu, rtol=0, atol=1e-10)
    # bordered Cholesky: var' = var - kn(x, xp)^2 / (var(xp) + tau2), kn the posterior covariance
    from scipy.linalg import solve_triangular
    Vc = solve_triangular(f["L"], matern52(X, Xc, ls, s2), lower=True)
    kn = matern52(Xc, Xc[i:i + 1], ls, s2)[:, 0] - Vc.T @ Vc[:, i]
    np.testing.assert_allclose(sd2 ** 2, sd ** 2 - kn ** 2 / (sd[i] ** 2 + t2), rtol=0, atol=1e-10)


def test_believer_first_pick_is_top_ehvi():
    w = make_workload(5, n=512, m=40)
    mask = np.ones(512, np.uint8)
    hyp = [dict(lengthscale=w["lengthscale"][j], signal_var=1.0, noise_var=w["noise_var"][j],
                prior_mean=0.0) for j in range(2)]
    picks, vals, _, _ = kriging_believer(w["X"], w["Y"], hyp, w["Xc"], mask, w["ref"], 3)
    assert len(set(picks.tolist())) == 3
    mu = np.empty((512, 2)); sd = np.empty((512, 2))
    for j in range(2):
        mu[:, j], sd[:, j] = gp_posterior(gp_fit(w["X"], w["Y"][:, j], **hyp[j]), w["Xc"].astype(np.float64))
    e = ehvi(mu, sd, nondominated(w["Y"], w["ref"]), w["ref"])
    assert picks[0] == int(np.lexsort((np.arange(512), -e))[0])


def test_believer_second_step_by_the_downdate():
    # The refit-from-scratch believer against another route to its second step:
    # the mean stays, the variance drops by the bordered (rank-one) downdate
    # sigma'^2 = sigma^2 - kn^2 / (sigma^2(x_p) + tau^2), kn the posterior
    # covariance with the pick, and the front gains the fantasy mu(x_p).
    from scipy.linalg import solve_triangular
    w = make_workload(5, n=512, m=40)
    mask = np.ones(512, np.uint8)
    mask[::7] = 0
    hyp = [dict(lengthscale=w["lengthscale"][j], signal_var=1.0, noise_var=w["noise_var"][j],
                prior_mean=0.0) for j in range(2)]
    picks, vals, mu_end, sd_end = kriging_believer(w["X"], w["Y"], hyp, w["Xc"], mask, w["ref"], 2)
    Xc = w["Xc"].astype(np.float64)
    p1 = int(picks[0])
    mu = np.empty((512, 2)); sd = np.empty((512, 2)); sd2 = np.empty((512, 2))
    for j in range(2):
        f = gp_fit(w["X"], w["Y"][:, j], **hyp[j])
        mu[:, j], sd[:, j] = gp_posterior(f, Xc)
        ls = hyp[j]["lengthscale"]
        Vc = solve_triangular(f["L"], matern52(w["X"], Xc, ls, 1.0), lower=True)
        kn = matern52(Xc, Xc[p1:p1 + 1], ls, 1.0)[:, 0] - Vc.T @ Vc[:, p1]
        sd2[:, j] = np.sqrt(np.maximum(sd[:, j] ** 2 - kn ** 2 / (sd[p1, j] ** 2 + hyp[j]["noise_var"]), 0.0))
    np.testing.assert_allclose(mu_end, mu, rtol=0, atol=1e-9)
    np.testing.assert_allclose(sd_end, sd2, rtol=0, atol=1e-9)
    e = ehvi(mu, sd2, nondominated(np.vstack([w["Y"], mu[p1]]), w["ref"]), w["ref"])
    e[mask == 0] = -np.inf
    e[p1] = -np.inf
    order = np.lexsort((np.arange(512), -e))
    assert e[order[0]] - e[order[1]] > 1e-9 * max(1.0, e[order[0]])  # a clear second pick
    assert int(picks[1]) == int(order[0])
    assert vals[1] == pytest.approx(e[order[0]], rel=1e-9)


def test_pipeline_tiny_runs():
    w = make_workload(1)
    r = score_pool(w)
    assert r["idx"].shape == (1,) and r["n_valid"] > 0
    assert np.all(r["sigma"] >= 0)
