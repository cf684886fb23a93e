"""Maximum-likelihood GP hyperparameters (Sec. 4.3: SCOOT learns the noise
level tau^2 by maximum likelihood; the signal variance and the lengthscales
are learned the same way here).

TEST INFRASTRUCTURE ONLY (see the package docstring).

theta = (log l_1 .. log l_d, log s^2, log tau^2).  With K = k_theta(X, X) +
tau^2 I on the (optionally warped) inputs and r = y - c:

  NLL(theta) = 1/2 r^T K^-1 r + 1/2 log det K + m/2 log(2 pi)
  dNLL/dtheta_j = -1/2 tr((alpha alpha^T - K^-1) dK/dtheta_j),  alpha = K^-1 r

with dK/dlog s^2 = K - tau^2 I, dK/dlog tau^2 = tau^2 I and, for the
lengthscales (D_k = (x_k - x'_k) / l_k, r the scaled distance):
  Matern-5/2: dk/dlog l_k = 5/3 s^2 (1 + sqrt5 r) exp(-sqrt5 r) D_k^2
  Matern-3/2: dk/dlog l_k = 3 s^2 exp(-sqrt3 r) D_k^2.
"""
import numpy as np
from scipy.optimize import minimize

from .gp import COVARIANCES, kumaraswamy_warp


def nll_and_grad(theta, X, y, kernel="matern52", warp=None, prior_mean=0.0):
    X = np.asarray(X, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    m, d = X.shape
    theta = np.asarray(theta, dtype=np.float64)
    ls = np.exp(theta[:d])
    s2 = np.exp(theta[d])
    tau2 = np.exp(theta[d + 1])
    Xw = X if warp is None else kumaraswamy_warp(X, warp[0], warp[1])
    Kf = COVARIANCES[kernel](Xw, Xw, ls, s2)
    K = Kf + tau2 * np.eye(m)
    L = np.linalg.cholesky(K)
    r = y - prior_mean
    alpha = np.linalg.solve(K, r)
    nll = 0.5 * r @ alpha + np.sum(np.log(np.diag(L))) + 0.5 * m * np.log(2 * np.pi)
    Kinv = np.linalg.inv(K)
    W = np.outer(alpha, alpha) - Kinv
    D2 = ((Xw[:, None, :] - Xw[None, :, :]) / ls) ** 2     # m x m x d
    rr = np.sqrt(D2.sum(-1))
    if kernel == "matern52":
        radial = 5.0 / 3.0 * s2 * (1 + np.sqrt(5.0) * rr) * np.exp(-np.sqrt(5.0) * rr)
    else:
        radial = 3.0 * s2 * np.exp(-np.sqrt(3.0) * rr)
    grad = np.empty(d + 2)
    for k in range(d):
        grad[k] = -0.5 * np.sum(W * radial * D2[:, :, k])
    grad[d] = -0.5 * np.sum(W * Kf)
    grad[d + 1] = -0.5 * tau2 * np.trace(W)
    return nll, grad


def warp_derivatives(X, a, b):
    """Kumaraswamy warp w = 1 - (1 - x^a)^b of every input (x clamped to [0, 1])
    and its derivatives in log a and log b:

      dw/dlog a = a b (1 - x^a)^(b - 1) x^a ln x,
      dw/dlog b = -b (1 - x^a)^b ln(1 - x^a),

    both 0 at x = 0 and x = 1 (their limits there)."""
    X = np.clip(np.asarray(X, dtype=np.float64), 0.0, 1.0)
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    inner = (X > 0) & (X < 1)
    Xi = np.where(inner, X, 0.5)
    u = Xi ** a
    w = 1.0 - (1.0 - X ** a) ** b
    da = np.where(inner, a * b * (1.0 - u) ** (b - 1.0) * u * np.log(Xi), 0.0)
    db = np.where(inner, -b * (1.0 - u) ** b * np.log(1.0 - u), 0.0)
    return w, da, db


def nll_and_grad_warp(theta, X, y, kernel="matern52", prior_mean=0.0):
    """The NLL with the input warping learned too (Sec. 4.3: Matern-3/2 with
    input warping after Snoek et al., whose warp parameters are fitted with
    the GP): theta = (log l_1..d, log s^2, log tau^2, log a_1..d, log b_1..d).

    The warped inputs w_ik enter K through the scaled distance only, and
    dk/dw_ik = -R_ij (w_ik - w_jk) / l_k^2 with R the radial factor of the
    lengthscale derivatives above (k'(r) / r = -R for both covariances), so

      dK_ij/dlog a_k = -R_ij (w_ik - w_jk) (g_ik - g_jk) / l_k^2,  g = dw/dlog a_k,

    and likewise for log b_k; the gradient is -1/2 tr(W dK/dtheta) as before.
    Returns (nll, gradient of length 3d + 2)."""
    X = np.asarray(X, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    m, d = X.shape
    theta = np.asarray(theta, dtype=np.float64)
    a, b = np.exp(theta[d + 2:2 * d + 2]), np.exp(theta[2 * d + 2:3 * d + 2])
    Xw, ga, gb = warp_derivatives(X, a, b)
    nll, g0 = nll_and_grad(theta[:d + 2], Xw, y, kernel, None, prior_mean)
    ls = np.exp(theta[:d])
    s2, tau2 = np.exp(theta[d]), np.exp(theta[d + 1])
    K = COVARIANCES[kernel](Xw, Xw, ls, s2) + tau2 * np.eye(m)
    alpha = np.linalg.solve(K, y - prior_mean)
    W = np.outer(alpha, alpha) - np.linalg.inv(K)
    diff = Xw[:, None, :] - Xw[None, :, :]                  # m x m x d
    rr = np.sqrt(np.sum((diff / ls) ** 2, axis=-1))
    if kernel == "matern52":
        radial = 5.0 / 3.0 * s2 * (1 + np.sqrt(5.0) * rr) * np.exp(-np.sqrt(5.0) * rr)
    else:
        radial = 3.0 * s2 * np.exp(-np.sqrt(3.0) * rr)
    grad = np.empty(3 * d + 2)
    grad[:d + 2] = g0
    for k in range(d):
        common = W * radial * diff[:, :, k] / ls[k] ** 2
        grad[d + 2 + k] = 0.5 * np.sum(common * (ga[:, None, k] - ga[None, :, k]))
        grad[2 * d + 2 + k] = 0.5 * np.sum(common * (gb[:, None, k] - gb[None, :, k]))
    return nll, grad


def fit_hyperparameters_warp(X, y, theta0, lower, upper, kernel="matern32", prior_mean=0.0):
    """Minimise the warped NLL over the box (3d + 2 log parameters) from theta0
    with scipy's L-BFGS-B.  Returns (theta, nll)."""
    res = minimize(lambda t: nll_and_grad_warp(t, X, y, kernel, prior_mean), np.asarray(theta0, np.float64),
                   jac=True, method="L-BFGS-B", bounds=list(zip(lower, upper)),
                   options=dict(maxiter=1000, ftol=1e-13, gtol=1e-9))
    return res.x, res.fun


def fit_hyperparameters(X, y, theta0, lower, upper, kernel="matern52", warp=None, prior_mean=0.0):
    """Minimise NLL over the box [lower, upper] (log parameters) from theta0
    with scipy's L-BFGS-B.  Returns (theta, nll)."""
    res = minimize(lambda t: nll_and_grad(t, X, y, kernel, warp, prior_mean), np.asarray(theta0, np.float64),
                   jac=True, method="L-BFGS-B", bounds=list(zip(lower, upper)),
                   options=dict(maxiter=500, ftol=1e-13, gtol=1e-9))
    return res.x, res.fun
