"""Small seeded search spaces and synthetic evaluators for the suggestion-step
tests (shared by the oracle pins and the GPU parity tests; no method
arithmetic here)."""
import numpy as np

from workloads.synth import sobol_table


def space(d=4, constrained=True):
    """d dims: continuous, continuous, a 5-level grid, a boolean, then more
    continuous ones; one known constraint x0 - x1 <= 0.3 (an order between
    two knobs, loosened)."""
    levels = [0, 0, 5, 1] + [0] * (d - 4)
    poly, vinit = sobol_table(d)
    sp = dict(levels=np.array(levels, np.int32), poly=poly, vinit=vinit)
    if constrained:
        A = np.zeros((1, d))
        A[0, 0], A[0, 1] = 1.0, -1.0
        sp.update(A=A, b=np.array([0.3]))
    return sp


def evaluate(X, p, seed=11):
    """Objective values (minimised) and validity: crashes where x0 + x2 > 1.4."""
    X = np.asarray(X, dtype=np.float64)
    rng = np.random.default_rng(seed)
    W = rng.uniform(0.5, 1.5, size=(p, X.shape[1]))
    Y = np.stack([np.sin(3.0 * X @ W[j]) + 0.3 * np.cos(5.0 * X[:, j % X.shape[1]]) for j in range(p)], axis=1)
    valid = (X[:, 0] + X[:, 2] <= 1.4).astype(np.uint8)
    return Y, valid


def observations(n_obs, d=4, p=1, seed=3):
    """Uniform configurations on the space's grids and their evaluation."""
    rng = np.random.default_rng(seed)
    X = rng.random((n_obs, d))
    X[:, 2] = np.rint(X[:, 2] * 4) / 4
    X[:, 3] = (X[:, 3] >= 0.5).astype(np.float64)
    X = X.astype(np.float32).astype(np.float64)
    Y, valid = evaluate(X, p)
    return X, Y, valid


def fixed_theta(p, d, ell=0.4, s2=1.0, tau2=1e-3):
    th = np.log(np.array([ell] * d + [s2, tau2]))
    return np.tile(th, (p, 1))
