"""Expected improvement, Sec. 4.4.1, Eq. 8, for a minimised objective.

The paper maximises f and writes EI(x) = E[max(0, f(x) + xi - f(x+))].  With
y = -f minimised and y* the best (lowest) observed feasible value this is

    EI(x) = E[max(0, y* + xi - Y)],   Y ~ N(mu(x), sigma(x)^2),

i.e. EI = G(y* + xi) with the partial expectation

    G(c) = E[(c - Y)^+] = (c - mu) Phi(u) + sigma phi(u),  u = (c - mu) / sigma,

and G(c) = max(0, c - mu) when sigma = 0.  The paper fixes xi = 1e-4 (Sec. 4.5.1)
and adds it to the improvement; ``xi`` is a signed argument.
"""
import numpy as np
from scipy.special import ndtr

XI_PAPER = 1e-4


def norm_pdf(u):
    return np.exp(-0.5 * u * u) / np.sqrt(2.0 * np.pi)


def partial_expectation(c, mu, sigma):
    """G(c) = E[(c - Y)^+] for Y ~ N(mu, sigma^2), elementwise; c may be +-inf."""
    c = np.asarray(c, dtype=np.float64)
    mu = np.asarray(mu, dtype=np.float64)
    sigma = np.asarray(sigma, dtype=np.float64)
    c, mu, sigma = np.broadcast_arrays(c, mu, sigma)
    out = np.zeros(c.shape)
    pos = sigma > 0
    fin = np.isfinite(c)
    m = pos & fin
    u = (c[m] - mu[m]) / sigma[m]
    out[m] = (c[m] - mu[m]) * ndtr(u) + sigma[m] * norm_pdf(u)
    z = (~pos) & fin
    out[z] = np.maximum(0.0, c[z] - mu[z])
    out[np.isposinf(c)] = np.inf
    return out


def expected_improvement(mu, sigma, best_y, xi=XI_PAPER):
    """Eq. 8 mirrored to minimisation: EI = G(best_y + xi)."""
    return partial_expectation(best_y + xi, mu, sigma)
