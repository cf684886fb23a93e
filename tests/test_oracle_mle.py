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


# ------------------------------------------ learning the input warping too
from oracle.mle import fit_hyperparameters_warp, nll_and_grad_warp, warp_derivatives  # noqa: E402


def test_warp_derivatives_at_the_identity_warp():
    """a = b = 1 is the identity: w = x, dw/dlog a = x ln x, dw/dlog b =
    -(1 - x) ln(1 - x), and both vanish at 0 and 1."""
    x = np.array([[0.0, 0.25, 0.5, 0.75, 1.0]]).T
    w, da, db = warp_derivatives(x, np.ones(1), np.ones(1))
    np.testing.assert_allclose(w[:, 0], x[:, 0], rtol=0, atol=1e-16)
    inner = x[1:4, 0]
    np.testing.assert_allclose(da[1:4, 0], inner * np.log(inner), rtol=1e-14)
    np.testing.assert_allclose(db[1:4, 0], -(1 - inner) * np.log(1 - inner), rtol=1e-14)
    assert da[0, 0] == da[4, 0] == db[0, 0] == db[4, 0] == 0.0
    # a = 2, b = 3 at 1/2: w = 37/64; dw/dlog a = 2*3*(3/4)^2*(1/4)*ln(1/2); dw/dlog b = -3 (3/4)^3 ln(3/4)
    w, da, db = warp_derivatives(np.array([[0.5]]), np.array([2.0]), np.array([3.0]))
    assert w[0, 0] == pytest.approx(37 / 64, rel=1e-15)
    assert da[0, 0] == pytest.approx(6 * 9 / 16 * 0.25 * np.log(0.5), rel=1e-14)
    assert db[0, 0] == pytest.approx(-3 * (27 / 64) * np.log(0.75), rel=1e-14)


@pytest.mark.parametrize("kernel", ["matern52", "matern32"])
def test_warp_gradient_matches_finite_differences(kernel):
    X, y = _data(4, m=24, d=3)
    X[0, 0], X[1, 1], X[2, 2] = 0.0, 1.0, 0.5        # endpoints and a grid value
    theta = np.log(np.array([0.4, 0.9, 0.5, 1.2, 0.02, 0.6, 1.0, 2.0, 1.5, 0.8, 1.0]))
    f0, g = nll_and_grad_warp(theta, X, y, kernel, prior_mean=0.05)
    h = 1e-6
    fd = np.array([(nll_and_grad_warp(theta + h * e, X, y, kernel, 0.05)[0] -
                    nll_and_grad_warp(theta - h * e, X, y, kernel, 0.05)[0]) / (2 * h) for e in np.eye(len(theta))])
    np.testing.assert_allclose(g, fd, rtol=1e-5, atol=1e-7)
    # at fixed warp parameters it is the NLL with that warp given
    f1, g1 = nll_and_grad(theta[:5], X, y, kernel, (np.exp(theta[5:8]), np.exp(theta[8:11])), prior_mean=0.05)
    assert f0 == pytest.approx(f1, rel=1e-13)
    np.testing.assert_allclose(g[:5], g1, rtol=1e-12, atol=1e-14)


def test_learned_warp_optimum_against_sklearn_on_prewarped_inputs():
    """At the optimum of the warped likelihood, sklearn's log marginal
    likelihood on the inputs pre-warped with the learned (a, b) is minus the
    NLL, and its gradient in (s^2, l, tau^2) vanishes where the optimum is
    inside the box; learning the warp does no worse than the identity warp."""
    rng = np.random.default_rng(7)
    X = rng.random((45, 2))
    y = np.sin(6 * X[:, 0] ** 3) + 0.5 * X[:, 1] ** 0.3 + 0.02 * rng.standard_normal(45)
    y = y - y.mean()
    d = 2
    lo = np.log(np.array([0.02] * d + [0.05, 1e-6] + [0.2] * (2 * d)))
    hi = np.log(np.array([10.0] * d + [20.0, 1.0] + [5.0] * (2 * d)))
    start = np.log(np.array([0.5] * d + [1.0, 1e-3] + [1.0] * (2 * d)))
    theta, f = fit_hyperparameters_warp(X, y, start, lo, hi, "matern32")
    a, b = np.exp(theta[d + 2:2 * d + 2]), np.exp(theta[2 * d + 2:])
    Xw = kumaraswamy_warp(X, a, b)
    gpr = GaussianProcessRegressor(ConstantKernel(1.0) * Matern(length_scale=np.ones(d), nu=1.5) + WhiteKernel(1.0),
                                   alpha=0.0, optimizer=None, normalize_y=False).fit(Xw, y)
    t_sk = np.concatenate([[theta[d]], theta[:d], [theta[d + 1]]])
    lml, g_sk = gpr.log_marginal_likelihood(t_sk, eval_gradient=True)
    assert f == pytest.approx(-lml, rel=1e-10)
    inner = np.concatenate([[theta[d]], theta[:d], [theta[d + 1]]])
    lo_sk = np.concatenate([[lo[d]], lo[:d], [lo[d + 1]]])
    hi_sk = np.concatenate([[hi[d]], hi[:d], [hi[d + 1]]])
    free = (inner > lo_sk + 1e-6) & (inner < hi_sk - 1e-6)
    assert np.all(np.abs(g_sk[free]) < 1e-4)
    _, g = nll_and_grad_warp(theta, X, y, "matern32")
    wfree = (theta[d + 2:] > lo[d + 2:] + 1e-6) & (theta[d + 2:] < hi[d + 2:] - 1e-6)
    assert np.all(np.abs(g[d + 2:][wfree]) < 1e-4)
    th0, f_id = fit_hyperparameters(X, y, start[:d + 2], lo[:d + 2], hi[:d + 2], "matern32")
    assert f <= f_id + 1e-9
