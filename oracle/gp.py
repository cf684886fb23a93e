"""Gaussian-process surrogate: the posterior of Sec. 4.3, Eq. 4 and Eq. 5.

TEST INFRASTRUCTURE ONLY (see the package docstring).

mu(x)      = c + k(x, X) (K + tau^2 I)^-1 (Y - c)
sigma^2(x) = k(x, x) - k(x, X) (K + tau^2 I)^-1 k(X, x)

with K = k(X, X).  Eq. 4 is written with zero prior mean; ``prior_mean`` c is
an explicit argument whose default 0 reproduces it.  The inverse is applied
through the Cholesky factor L of K + tau^2 I: alpha = L^-T L^-1 (Y - c) and
sigma^2 = k(x, x) - ||L^-1 k(X, x)||^2, which are the same quantities.
Independent outputs (Sec. 4.3, last paragraph) are independent calls.

Covariances: Matern-5/2 ARD (the workloads' kernel) and the paper's own,
Matern-3/2 with input warping (Sec. 4.3, after Snoek et al., "Input warping
for Bayesian optimization of non-stationary functions"): every input
dimension in [0, 1] passes through the Kumaraswamy distribution function
w(x) = 1 - (1 - x^a)^b (a, b > 0, one pair per dimension) before the
covariance sees it.
"""
import numpy as np
from scipy.linalg import solve_triangular

SQRT5 = np.sqrt(5.0)
SQRT3 = np.sqrt(3.0)


def matern52(A, B, lengthscale, signal_var):
    """Matern-5/2 ARD covariance between the rows of A (a x d) and B (b x d).

    k(x, x') = s^2 (1 + sqrt5 r + 5 r^2 / 3) exp(-sqrt5 r),
    r^2 = sum_k ((x_k - x'_k) / l_k)^2.
    """
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    ls = np.asarray(lengthscale, dtype=np.float64)
    diff = (A[:, None, :] - B[None, :, :]) / ls
    r = np.sqrt(np.sum(diff * diff, axis=-1))
    return signal_var * (1.0 + SQRT5 * r + 5.0 / 3.0 * r * r) * np.exp(-SQRT5 * r)


def matern32(A, B, lengthscale, signal_var):
    """Matern-3/2 ARD covariance: k(x, x') = s^2 (1 + sqrt3 r) exp(-sqrt3 r)."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    ls = np.asarray(lengthscale, dtype=np.float64)
    diff = (A[:, None, :] - B[None, :, :]) / ls
    r = np.sqrt(np.sum(diff * diff, axis=-1))
    return signal_var * (1.0 + SQRT3 * r) * np.exp(-SQRT3 * r)


COVARIANCES = {"matern52": matern52, "matern32": matern32}


def kumaraswamy_warp(X, a, b):
    """w(x) = 1 - (1 - x^a)^b per dimension, x clamped to [0, 1]."""
    X = np.clip(np.asarray(X, dtype=np.float64), 0.0, 1.0)
    return 1.0 - (1.0 - X ** np.asarray(a, dtype=np.float64)) ** np.asarray(b, dtype=np.float64)


def gp_fit(X, y, lengthscale, signal_var, noise_var, prior_mean=0.0, kernel="matern52", warp=None):
    """Factor K + tau^2 I and solve for the weights of Eq. 4.

    ``kernel`` is "matern52" or "matern32"; ``warp`` is None or (a, b), two
    arrays of d positive Kumaraswamy parameters applied to every input.
    Returns a dict with the inputs and L (lower Cholesky factor), alpha.
    Raises numpy.linalg.LinAlgError when K + tau^2 I is not positive definite.
    """
    X = np.asarray(X, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    Xw = X if warp is None else kumaraswamy_warp(X, warp[0], warp[1])
    K = COVARIANCES[kernel](Xw, Xw, lengthscale, signal_var) + noise_var * np.eye(len(X))
    L = np.linalg.cholesky(K)
    resid = y - prior_mean
    alpha = solve_triangular(L.T, solve_triangular(L, resid, lower=True), lower=False)
    return dict(X=X, Xw=Xw, y=y, lengthscale=np.asarray(lengthscale, dtype=np.float64),
                signal_var=float(signal_var), noise_var=float(noise_var),
                prior_mean=float(prior_mean), L=L, alpha=alpha, K=K, kernel=kernel, warp=warp)


def _cross(fit, Xc):
    Xcw = Xc if fit.get("warp") is None else kumaraswamy_warp(Xc, fit["warp"][0], fit["warp"][1])
    cov = COVARIANCES[fit.get("kernel", "matern52")]
    return cov(Xcw, fit.get("Xw", fit["X"]), fit["lengthscale"], fit["signal_var"])


def gp_posterior(fit, Xc, chunk=8192):
    """Posterior mean and standard deviation of the latent f at the rows of Xc.

    Eq. 4 for mu, Eq. 5 for sigma^2; sigma^2 below zero (rounding) is clamped.
    """
    Xc = np.asarray(Xc, dtype=np.float64)
    n = len(Xc)
    mu = np.empty(n)
    sigma = np.empty(n)
    for s in range(0, n, chunk):
        Ks = _cross(fit, Xc[s:s + chunk])
        mu[s:s + chunk] = fit["prior_mean"] + Ks @ fit["alpha"]
        V = solve_triangular(fit["L"], Ks.T, lower=True)
        var = fit["signal_var"] - np.sum(V * V, axis=0)
        sigma[s:s + chunk] = np.sqrt(np.maximum(var, 0.0))
    return mu, sigma


def gp_posterior_var_direct(fit, Xc):
    """Eq. 5 with an explicit inverse, for tiny inputs: a second route to sigma^2."""
    Ks = _cross(fit, np.asarray(Xc, dtype=np.float64))
    Kinv = np.linalg.inv(fit["K"])
    return fit["signal_var"] - np.einsum("ij,jk,ik->i", Ks, Kinv, Ks)
