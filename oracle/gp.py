"""Gaussian-process surrogate: the posterior of Sec. 4.3, Eq. 4 and Eq. 5.

mu(x)      = c + k(x, X) (K + tau^2 I)^-1 (Y - c)
sigma^2(x) = k(x, x) - k(x, X) (K + tau^2 I)^-1 k(X, x)

with K = k(X, X).  Eq. 4 is written with zero prior mean; ``prior_mean`` c is
an explicit argument whose default 0 reproduces it.  The inverse is applied
through the Cholesky factor L of K + tau^2 I: alpha = L^-T L^-1 (Y - c) and
sigma^2 = k(x, x) - ||L^-1 k(X, x)||^2, which are the same quantities.
Independent outputs (Sec. 4.3, last paragraph) are independent calls.
"""
import numpy as np
from scipy.linalg import solve_triangular

SQRT5 = np.sqrt(5.0)


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


def gp_fit(X, y, lengthscale, signal_var, noise_var, prior_mean=0.0):
    """Factor K + tau^2 I and solve for the weights of Eq. 4.

    Returns a dict with the inputs and L (lower Cholesky factor), alpha.
    Raises numpy.linalg.LinAlgError when K + tau^2 I is not positive definite.
    """
    X = np.asarray(X, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    K = matern52(X, X, lengthscale, signal_var) + noise_var * np.eye(len(X))
    L = np.linalg.cholesky(K)
    resid = y - prior_mean
    alpha = solve_triangular(L.T, solve_triangular(L, resid, lower=True), lower=False)
    return dict(X=X, y=y, lengthscale=np.asarray(lengthscale, dtype=np.float64),
                signal_var=float(signal_var), noise_var=float(noise_var),
                prior_mean=float(prior_mean), L=L, alpha=alpha, K=K)


def gp_posterior(fit, Xc, chunk=8192):
    """Posterior mean and standard deviation of the latent f at the rows of Xc.

    Eq. 4 for mu, Eq. 5 for sigma^2; sigma^2 below zero (rounding) is clamped.
    """
    Xc = np.asarray(Xc, dtype=np.float64)
    n = len(Xc)
    mu = np.empty(n)
    sigma = np.empty(n)
    for s in range(0, n, chunk):
        Ks = matern52(Xc[s:s + chunk], fit["X"], fit["lengthscale"], fit["signal_var"])
        mu[s:s + chunk] = fit["prior_mean"] + Ks @ fit["alpha"]
        V = solve_triangular(fit["L"], Ks.T, lower=True)
        var = fit["signal_var"] - np.sum(V * V, axis=0)
        sigma[s:s + chunk] = np.sqrt(np.maximum(var, 0.0))
    return mu, sigma


def gp_posterior_var_direct(fit, Xc):
    """Eq. 5 with an explicit inverse, for tiny inputs: a second route to sigma^2."""
    Ks = matern52(Xc, fit["X"], fit["lengthscale"], fit["signal_var"])
    Kinv = np.linalg.inv(fit["K"])
    return fit["signal_var"] - np.einsum("ij,jk,ik->i", Ks, Kinv, Ks)
