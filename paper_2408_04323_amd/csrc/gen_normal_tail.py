"""Coefficients of the rational approximation used by the fp32 acquisition
kernels for the normal partial expectation.

For x >= 0 let M(x) = P(Z > x) / phi(x) (the Mills ratio of the standard
normal) and g(x) = 1 - x M(x), so that h(-x) = phi(x) g(x) with
h(u) = u Phi(u) + phi(u).  g falls from 1 at 0 like 1 / x^2; it is fitted on
[0, 14] by R(s) = P4(s) / Q6(s), s = x / 4 (the denominator two degrees higher
to follow the 1 / x^2 tail), minimising the relative error: linearised least
squares iterated on the previous denominator (Sanathanan-Koerner), then
reweighted towards the largest errors (Lawson).  Prints the two coefficient
lists and the achieved relative error in double and in float32 Horner
evaluation.  Run: python gen_normal_tail.py
"""
import numpy as np
from scipy.special import erfcx

SCALE = 4.0
X_MAX = 14.0
DEG_P, DEG_Q = 4, 6


def g_exact(x):
    return 1.0 - x * erfcx(x / np.sqrt(2.0)) * np.sqrt(np.pi / 2.0)


def fit():
    x = np.concatenate([np.linspace(0.0, 1.0, 2000), np.linspace(1.0, X_MAX, 20000)[1:]])
    y = g_exact(x)
    s = x / SCALE
    w = 1.0 / y
    q_prev = np.ones_like(x)
    for it in range(80):
        A = np.hstack([np.vander(s, DEG_P + 1, increasing=True),
                       -y[:, None] * np.vander(s, DEG_Q + 1, increasing=True)[:, 1:]])
        W = (w / q_prev)[:, None]
        c, *_ = np.linalg.lstsq(A * W, y * W[:, 0], rcond=None)
        p = c[:DEG_P + 1]
        q = np.concatenate([[1.0], c[DEG_P + 1:]])
        q_prev = np.polyval(q[::-1], s)
        err = (np.polyval(p[::-1], s) / q_prev - y) / y
        if it > 20:
            w = w * (1.0 + 50.0 * np.abs(err) / np.max(np.abs(err)))
    return x, y, p, q, np.max(np.abs(err))


def eval_f32(p, q, x):
    s = (x.astype(np.float32) * np.float32(1.0 / SCALE)).astype(np.float32)
    P = np.float32(p[-1])
    for c in p[-2::-1]:
        P = (P * s + np.float32(c)).astype(np.float32)
    Q = np.float32(q[-1])
    for c in q[-2::-1]:
        Q = (Q * s + np.float32(c)).astype(np.float32)
    return (P / Q).astype(np.float32)


if __name__ == "__main__":
    x, y, p, q, e = fit()
    e32 = np.max(np.abs((eval_f32(p, q, x).astype(np.float64) - y) / y))
    assert np.min(np.polyval(q[::-1], x / SCALE)) >= 1.0
    print("P:", ", ".join(f"{v:.9e}f" for v in p))
    print("Q:", ", ".join(f"{v:.9e}f" for v in q))
    print(f"max relative error on [0, {X_MAX}]: double {e:.2e}, float32 Horner {e32:.2e}")
