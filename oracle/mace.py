"""MACE suggestion for one objective (Sec. 4.5.1, with Eq. 6-8 and the
parallel pick of Sec. 4.6), objective minimised.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper scores every candidate with three acquisition functions, takes the
candidates on the Pareto front of the three scores (all maximised) and
suggests k of them drawn at random.  With y = -f minimised, y* the best
observed feasible value and Y ~ N(mu, sigma^2):

* UCB (Eq. 6): the paper's mu(f) + beta sigma(f) becomes the score
  beta * sigma - mu (the mean of -Y plus beta standard deviations);
* PI (Eq. 7): P(f(x) + xi > f(x+)) becomes P(Y < y* + xi)
  = Phi((y* + xi - mu) / sigma), and 1 or 0 (is mu < y* + xi) when sigma = 0;
* EI (Eq. 8): E[(y* + xi - Y)^+], as in ``acquisition``.

beta of the t-th tuning iteration: 2 log(t^2 pi^2 / (6 delta)) with
delta = 1 / t^2.  The paper multiplies sigma by this beta itself (Eq. 6 and
the schedule both name it beta); the cited GP-UCB rule multiplies by its
square root.  The oracle follows the paper's text and takes the multiplier as
an argument either way.

Front: a candidate is dominated when another eligible candidate scores at
least as high on all three and strictly higher on one; the front is the set of
eligible candidates no other eligible candidate dominates (equal score vectors
do not dominate each other).  Eligible = mask non-zero and no NaN score.

Random pick: the draw comes from a counter-based generator so that any device
can reproduce it: u_i, the i-th output (i = 0, 1, ...) of SplitMix64 started
from ``seed`` (Steele, Lea and Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014; the variant with Stafford's 64-bit finaliser), is
candidate i's draw, and the pick is the q front members with the largest u_i
(index ascending on equal draws).  Ranking i.i.d. uniform draws yields a
uniformly random q-subset of the front, in random order.  A front smaller than
q leaves -1 in the tail.
"""
import numpy as np
from scipy.special import ndtr

from .acquisition import expected_improvement

MASK64 = (1 << 64) - 1
GOLDEN_GAMMA = 0x9E3779B97F4A7C15  # odd integer nearest 2^64 / golden ratio
MIX_M1 = 0xBF58476D1CE4E5B9
MIX_M2 = 0x94D049BB133111EB


def ucb_beta(t):
    """beta_t = 2 log(t^2 pi^2 / (6 delta)) with delta = 1 / t^2 (Sec. 4.5.1)."""
    t = float(t)
    delta = 1.0 / (t * t)
    return 2.0 * np.log(t * t * np.pi ** 2 / (6.0 * delta))


def ucb_score(mu, sigma, beta):
    """Eq. 6 for -Y: beta * sigma - mu."""
    return beta * np.asarray(sigma, dtype=np.float64) - np.asarray(mu, dtype=np.float64)


def probability_of_improvement(mu, sigma, best_y, xi):
    """Eq. 7 for a minimised objective: P(Y < best_y + xi)."""
    mu = np.asarray(mu, dtype=np.float64)
    sigma = np.asarray(sigma, dtype=np.float64)
    c = best_y + xi
    out = np.where(mu < c, 1.0, 0.0)
    pos = sigma > 0
    out[pos] = ndtr((c - mu[pos]) / sigma[pos])
    return out


def mace_scores(mu, sigma, best_y, xi, beta):
    """(ucb, pi, ei), each (n,)."""
    return (ucb_score(mu, sigma, beta), probability_of_improvement(mu, sigma, best_y, xi),
            expected_improvement(mu, sigma, best_y, xi))


def pareto_front_max(scores, mask=None):
    """scores: (n, k) maximised.  Returns a bool (n,) array: eligible and not
    dominated by any eligible candidate.  Brute force over candidates."""
    S = np.asarray(scores, dtype=np.float64)
    n = len(S)
    ok = ~np.isnan(S).any(axis=1)
    if mask is not None:
        ok &= np.asarray(mask) != 0
    E = S[ok]
    front = np.zeros(n, dtype=bool)
    for i in np.flatnonzero(ok):
        ge = (E >= S[i]).all(axis=1)
        gt = (E > S[i]).any(axis=1)
        front[i] = not (ge & gt).any()
    return front


def splitmix64_mix(z):
    """Stafford's 64-bit finaliser as used by SplitMix64 (Python ints)."""
    z = (z ^ (z >> 30)) * MIX_M1 & MASK64
    z = (z ^ (z >> 27)) * MIX_M2 & MASK64
    return z ^ (z >> 31)


def splitmix64(seed, i):
    """Output number i (0-based) of SplitMix64 started from ``seed``: the state
    after i + 1 increments by the golden gamma, finalised."""
    return splitmix64_mix((seed + (i + 1) * GOLDEN_GAMMA) & MASK64)


def random_pick(flags, seed, q):
    """The q flagged candidates with the largest SplitMix64 draw (index
    ascending on equal draws).  Returns (idx int64 (q,), n_flagged)."""
    cand = np.flatnonzero(np.asarray(flags) != 0)
    draws = [splitmix64(seed, int(i)) for i in cand]
    order = sorted(range(len(cand)), key=lambda k: (-draws[k], int(cand[k])))
    idx = np.full(q, -1, dtype=np.int64)
    for r, k in enumerate(order[:q]):
        idx[r] = cand[k]
    return idx, len(cand)


def mace_suggest(mu, sigma, mask, best_y, xi, beta, seed, q):
    """Scores, front and pick for one objective.  Returns a dict."""
    ucb, pi, ei = mace_scores(mu, sigma, best_y, xi, beta)
    front = pareto_front_max(np.stack([ucb, pi, ei], axis=1), mask)
    idx, n_front = random_pick(front, seed, q)
    return dict(ucb=ucb, pi=pi, ei=ei, front=front, idx=idx, n_front=n_front)
