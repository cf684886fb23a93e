"""Pins of the maximum-likelihood oracle (Sec. 4.3) to sklearn's log marginal
likelihood and its gradient, and to finite differences."""
import numpy as np
import pytest
from sklearn.gaussian_process import GaussianProcessRegressor
from sklearn.gaussian_process.kernels import ConstantKernel, Matern, WhiteKernel

from oracle.gp import kumaraswamy_warp
from oracle.mle import fit_hyperparameters, nll_and_grad


def _data(seed, m=30, d=3):
    rng = np.random.default_rng(seed)
    X = rng.random((m, d))
    y = np.sin(4 * X[:, 0]) + X[:, 1] ** 2 + 0.05 * rng.standard_normal(m)
    return X, y - y.mean()


@pytest.mark.parametrize("kernel,nu", [("matern52", 2.5), ("matern32", 1.5)])
def test_nll_and_gradient_match_sklearn(kernel, nu):
    X, y = _data(1)
    theta = np.log(np.array([0.3, 0.7, 1.4, 0.8, 0.02]))
    nll, g = nll_and_grad(theta, X, y, kernel)
    # alpha = 0: no extra jitter on the diagonal (the white kernel carries tau^2)
    gpr = GaussianProcessRegressor(ConstantKernel(1.0) * Matern(length_scale=np.ones(3), nu=nu) + WhiteKernel(1.0),
                                   alpha=0.0, optimizer=None, normalize_y=False).fit(X, y)
    # sklearn's theta: [log s2, log l_1..l_d, log tau2]
    t_sk = np.concatenate([[theta[3]], theta[:3], [theta[4]]])
    lml, g_sk = gpr.log_marginal_likelihood(t_sk, eval_gradient=True)
    assert nll == pytest.approx(-lml, rel=1e-12)
    np.testing.assert_allclose(g, -np.concatenate([g_sk[1:4], [g_sk[0]], [g_sk[4]]]), rtol=1e-8, atol=1e-10)


@pytest.mark.parametrize("kernel", ["matern52", "matern32"])
def test_gradient_matches_finite_differences_with_warping(kernel):
    X, y = _data(2, m=25, d=4)
    warp = (np.array([0.6, 1.0, 2.0, 1.3]), np.array([1.5, 0.8, 1.0, 2.2]))
    theta = np.log(np.array([0.4, 0.9, 0.5, 1.1, 1.3, 0.01]))
    f0, g = nll_and_grad(theta, X, y, kernel, warp, prior_mean=0.1)
    h = 1e-6
    fd = np.array([(nll_and_grad(theta + h * e, X, y, kernel, warp, 0.1)[0] -
                    nll_and_grad(theta - h * e, X, y, kernel, warp, 0.1)[0]) / (2 * h) for e in np.eye(6)])
    np.testing.assert_allclose(g, fd, rtol=1e-5, atol=1e-7)
    # warping acts through the inputs only: the warped NLL is the plain NLL on warped inputs
    f1, _ = nll_and_grad(theta, kumaraswamy_warp(X, *warp), y, kernel, None, prior_mean=0.1)
    assert f0 == pytest.approx(f1, rel=1e-14)


def test_fit_reaches_a_stationary_point_and_beats_the_start():
    X, y = _data(3, m=40, d=3)
    theta0 = np.log(np.array([0.5, 0.5, 0.5, 1.0, 0.1]))
    lo = np.log(np.array([0.05] * 3 + [0.05, 1e-6]))
    hi = np.log(np.array([5.0] * 3 + [20.0, 1.0]))
    theta, f = fit_hyperparameters(X, y, theta0, lo, hi)
    f0, _ = nll_and_grad(theta0, X, y)
    assert f < f0 - 1.0
    _, g = nll_and_grad(theta, X, y)
    interior = (theta > lo + 1e-6) & (theta < hi - 1e-6)
    assert np.all(np.abs(g[interior]) < 1e-4)
