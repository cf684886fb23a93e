"""Pins of the GP oracle (Sec. 4.3, Eq. 4-5) to facts outside the oracle."""
import numpy as np
import pytest
from sklearn.gaussian_process import GaussianProcessRegressor
from sklearn.gaussian_process.kernels import ConstantKernel, Matern

from oracle.gp import gp_fit, gp_posterior, gp_posterior_var_direct, matern52


def _data(seed, m=24, d=5):
    rng = np.random.default_rng(seed)
    X = rng.random((m, d))
    y = np.sin(3 * X).sum(axis=1) + 0.05 * rng.standard_normal(m)
    ls = rng.uniform(0.3, 1.2, size=d)
    return X, y, ls


def test_matern52_matches_sklearn():
    rng = np.random.default_rng(0)
    A, B = rng.random((7, 4)), rng.random((9, 4))
    ls = np.array([0.2, 0.5, 1.0, 2.0])
    ref = (ConstantKernel(1.7, "fixed") * Matern(length_scale=ls, nu=2.5))(A, B)
    got = matern52(A, B, ls, 1.7)
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=0)
    assert np.allclose(np.diag(matern52(A, A, ls, 1.7)), 1.7, rtol=0, atol=1e-15)


def test_matern52_scalar_closed_form():
    # one dimension, r = |x - x'| / l = 2: k = s2 (1 + 2 sqrt5 + 20/3) exp(-2 sqrt5)
    got = matern52(np.array([[0.0]]), np.array([[1.0]]), [0.5], 2.0)[0, 0]
    s5 = np.sqrt(5.0)
    assert got == pytest.approx(2.0 * (1 + 2 * s5 + 20 / 3) * np.exp(-2 * s5), rel=1e-15)


def test_fit_factor_and_weights():
    X, y, ls = _data(1)
    f = gp_fit(X, y, ls, 1.3, 1e-3, prior_mean=0.2)
    K = f["K"]
    assert np.linalg.norm(f["L"] @ f["L"].T - K) <= 1e-12 * np.linalg.norm(K)
    np.testing.assert_allclose(K @ f["alpha"], y - 0.2, rtol=0, atol=1e-9)


def test_posterior_matches_sklearn():
    X, y, ls = _data(2)
    rng = np.random.default_rng(3)
    Xc = rng.random((300, X.shape[1]))
    tau2 = 1e-3
    gpr = GaussianProcessRegressor(ConstantKernel(1.0, "fixed") * Matern(length_scale=ls, nu=2.5),
                                   alpha=tau2, optimizer=None, normalize_y=False).fit(X, y)
    mu_ref, sd_ref = gpr.predict(Xc, return_std=True)
    mu, sd = gp_posterior(gp_fit(X, y, ls, 1.0, tau2), Xc)
    np.testing.assert_allclose(mu, mu_ref, rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(sd, sd_ref, rtol=1e-7, atol=1e-9)


def test_single_observation_closed_form():
    # m = 1: mu = c + k(x,x1)(y1-c)/(s2+tau2), var = s2 - k(x,x1)^2/(s2+tau2)
    x1, y1, s2, t2, c = np.array([[0.3, 0.7]]), np.array([1.5]), 0.8, 0.05, 0.25
    ls = [0.4, 0.9]
    Xc = np.array([[0.3, 0.7], [0.5, 0.1], [0.9, 0.9]])
    k = matern52(Xc, x1, ls, s2)[:, 0]
    mu, sd = gp_posterior(gp_fit(x1, y1, ls, s2, t2, c), Xc)
    np.testing.assert_allclose(mu, c + k * (y1[0] - c) / (s2 + t2), rtol=1e-14)
    np.testing.assert_allclose(sd ** 2, s2 - k ** 2 / (s2 + t2), rtol=1e-13)


def test_noise_free_interpolation():
    X = np.array([[0.0, 0.0], [1.0, 0.0], [0.0, 1.0], [1.0, 1.0],
                  [0.5, 0.5], [0.5, 0.0], [0.0, 0.5], [1.0, 0.5]])
    y = np.array([0.3, -1.0, 2.0, 0.5, 1.1, -0.2, 0.7, 0.0])
    f = gp_fit(X, y, [0.3, 0.3], 1.0, 0.0)
    mu, sd = gp_posterior(f, X)
    assert np.max(np.abs(mu - y)) <= 1e-8
    assert np.max(sd ** 2) <= 1e-8


def test_variance_bounds_and_monotonicity():
    X, y, ls = _data(4)
    s2, t2 = 1.0, 1e-3
    f = gp_fit(X, y, ls, s2, t2)
    _, sd_obs = gp_posterior(f, X)
    assert np.all(sd_obs ** 2 <= s2 * t2 / (s2 + t2) + 1e-12)
    rng = np.random.default_rng(5)
    Xc = rng.random((500, X.shape[1]))
    _, sd = gp_posterior(f, Xc)
    assert np.all(sd ** 2 >= 0) and np.all(sd ** 2 <= s2 + 1e-12)
    # one more observation never raises the variance
    f2 = gp_fit(np.vstack([X, Xc[:1]]), np.append(y, 0.0), ls, s2, t2)
    _, sd2 = gp_posterior(f2, Xc)
    assert np.all(sd2 <= sd + 1e-12)
    # far from the data: prior mean and variance
    mu_far, sd_far = gp_posterior(gp_fit(X, y, ls, s2, t2, prior_mean=0.7), X[:3] + 100.0)
    np.testing.assert_allclose(mu_far, 0.7, atol=1e-12)
    np.testing.assert_allclose(sd_far ** 2, s2, atol=1e-12)


def test_variance_two_routes():
    X, y, ls = _data(6, m=12)
    f = gp_fit(X, y, ls, 1.0, 1e-2)
    Xc = np.random.default_rng(7).random((50, X.shape[1]))
    _, sd = gp_posterior(f, Xc)
    np.testing.assert_allclose(sd ** 2, gp_posterior_var_direct(f, Xc), rtol=1e-9, atol=1e-12)


def test_not_positive_definite_raises():
    X = np.zeros((3, 2))
    with pytest.raises(np.linalg.LinAlgError):
        gp_fit(X, np.zeros(3), [1.0, 1.0], 1.0, 0.0)


# ------------------------------------------- the paper's kernel: Matern-3/2 + warping
from oracle.gp import kumaraswamy_warp, matern32  # noqa: E402


def test_matern32_matches_sklearn():
    rng = np.random.default_rng(4)
    A, B = rng.random((7, 4)), rng.random((9, 4))
    ls = np.array([0.2, 0.5, 1.0, 2.0])
    ref = (ConstantKernel(0.6, "fixed") * Matern(length_scale=ls, nu=1.5))(A, B)
    np.testing.assert_allclose(matern32(A, B, ls, 0.6), ref, rtol=1e-13, atol=0)


def test_matern32_scalar_closed_form():
    # r = 2: k = s2 (1 + 2 sqrt3) exp(-2 sqrt3)
    got = matern32(np.array([[0.0]]), np.array([[1.0]]), [0.5], 2.0)[0, 0]
    s3 = np.sqrt(3.0)
    assert got == pytest.approx(2.0 * (1 + 2 * s3) * np.exp(-2 * s3), rel=1e-15)


def test_kumaraswamy_hand_values_and_special_cases():
    # a = 2, b = 3, x = 1/2: 1 - (1 - 1/4)^3 = 1 - 27/64 = 37/64
    assert kumaraswamy_warp(np.array([[0.5]]), [2.0], [3.0])[0, 0] == pytest.approx(37 / 64, rel=1e-15)
    x = np.linspace(0, 1, 101)[:, None]
    np.testing.assert_allclose(kumaraswamy_warp(x, [1.0], [1.0]), x, atol=1e-15)        # identity
    np.testing.assert_allclose(kumaraswamy_warp(x, [1.0], [2.5]), 1 - (1 - x) ** 2.5, atol=1e-15)
    np.testing.assert_allclose(kumaraswamy_warp(x, [0.4], [1.0]), x ** 0.4, atol=1e-15)
    w = kumaraswamy_warp(x, [0.7], [1.9])[:, 0]
    assert w[0] == 0.0 and w[-1] == 1.0 and np.all(np.diff(w) > 0)
    # outside the unit interval the input is clamped
    np.testing.assert_array_equal(kumaraswamy_warp(np.array([[-0.2], [1.3]]), [2.0], [0.5])[:, 0], [0.0, 1.0])


def test_warped_matern32_posterior_matches_sklearn_on_warped_inputs():
    X, y, ls = _data(6, m=30, d=4)
    rng = np.random.default_rng(7)
    Xc = rng.random((200, 4))
    a = np.array([0.5, 1.0, 2.0, 1.5])
    b = np.array([2.0, 0.7, 1.0, 1.2])
    tau2 = 1e-3
    gpr = GaussianProcessRegressor(ConstantKernel(0.9, "fixed") * Matern(length_scale=ls, nu=1.5),
                                   alpha=tau2, optimizer=None, normalize_y=False)
    # by hand: 1 - (1 - x^a)^b per column
    Xw = 1 - (1 - X ** a) ** b
    Xcw = 1 - (1 - Xc ** a) ** b
    mu_ref, sd_ref = gpr.fit(Xw, y).predict(Xcw, return_std=True)
    mu, sd = gp_posterior(gp_fit(X, y, ls, 0.9, tau2, kernel="matern32", warp=(a, b)), Xc)
    np.testing.assert_allclose(mu, mu_ref, rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(sd, sd_ref, rtol=1e-7, atol=1e-9)
    # the warp changes the answer (the test would pass vacuously otherwise)
    mu0, _ = gp_posterior(gp_fit(X, y, ls, 0.9, tau2, kernel="matern32"), Xc)
    assert np.max(np.abs(mu0 - mu)) > 1e-3
