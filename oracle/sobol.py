"""Candidate generation: a Sobol quasi-Monte Carlo pool with the search
space's grids, and the known constraints (Sec. 4.5.3: the solver's space is
pruned by known constraints; Sec. 4.7: a shortfall of suggestions is filled
with Sobol points; Sec. 4.1 and Algorithm 1: the first observations are
Sobol points).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sobol sequence (Sobol 1967; construction of Bratley and Fox 1988): dimension j
has a primitive polynomial over GF(2), x^s + a_1 x^(s-1) + ... + a_(s-1) x + 1,
given as the integer whose bits are its coefficients, and initial odd
integers m_1 .. m_s (m_k < 2^k).  For k > s,

  m_k = 2 a_1 m_(k-1) ^ 2^2 a_2 m_(k-2) ^ ... ^ 2^(s-1) a_(s-1) m_(k-s+1) ^ 2^s m_(k-s) ^ m_(k-s)

and the direction numbers are V_k = m_k 2^(32 - k) (32-bit).  Point i is the
XOR of V_k over the set bits k (1-based) of its Gray code i ^ (i >> 1), over
2^32 (Antonov and Saleev's ordering).  A polynomial of degree 0 (the integer
1) gives m_k = 1, the van der Corput sequence.

Grids: a dimension with level count L >= 2 is rounded to k / (L - 1)
(half to even, in double); L = 1 marks a boolean, 1 when x >= 1/2; L = 0 is
continuous.  Known constraints: a candidate is admissible when A x <= b holds
row by row, each row summed in double over k = 0 .. d-1 in order, every
product and sum rounded on its own (so that a boundary case is decided the
same way by any implementation that keeps that order).
"""
import numpy as np


def direction_numbers(poly, vinit, bits=32):
    """V [bits] (Python ints) of one dimension."""
    s = int(poly).bit_length() - 1
    m = [0] * (bits + 1)
    for k in range(1, bits + 1):
        if s == 0:
            m[k] = 1
        elif k <= s:
            m[k] = int(vinit[k - 1])
        else:
            v = m[k - s] ^ (m[k - s] << s)
            for t in range(1, s):
                a_t = (int(poly) >> (s - t)) & 1
                if a_t:
                    v ^= m[k - t] << t
            m[k] = v
    return [m[k] << (bits - k) for k in range(1, bits + 1)]


def sobol_points(poly, vinit, n, skip=0):
    """(n, d) float64 points i = skip .. skip + n - 1 (exact binary fractions)."""
    d = len(poly)
    V = [direction_numbers(poly[j], vinit[j]) for j in range(d)]
    out = np.zeros((n, d))
    for r in range(n):
        i = skip + r
        g = i ^ (i >> 1)
        for j in range(d):
            x = 0
            k = 0
            while g >> k:
                if (g >> k) & 1:
                    x ^= V[j][k]
                k += 1
            out[r, j] = x / 2.0 ** 32
    return out


def snap_levels(U, levels):
    X = np.array(U, dtype=np.float64, copy=True)
    for j, L in enumerate(levels):
        if L == 1:
            X[:, j] = (X[:, j] >= 0.5).astype(np.float64)
        elif L >= 2:
            X[:, j] = np.rint(X[:, j] * (L - 1)) / (L - 1)
    return X


def sobol_pool(poly, vinit, levels, n, skip=0):
    """The candidate pool: snapped Sobol points as float32 (n, d)."""
    return snap_levels(sobol_points(poly, vinit, n, skip), levels).astype(np.float32)


def known_constraints_mask(Xc, A, b):
    """uint8 (n,): 1 where every row of A x <= b holds."""
    X = np.asarray(Xc, dtype=np.float32).astype(np.float64)
    A = np.asarray(A, dtype=np.float64).reshape(-1, X.shape[1])
    b = np.asarray(b, dtype=np.float64)
    ok = np.ones(len(X), dtype=bool)
    for r in range(len(A)):
        s = np.zeros(len(X))
        for k in range(X.shape[1]):
            s = s + A[r, k] * X[:, k]
        ok &= s <= b[r]
    return ok.astype(np.uint8)
