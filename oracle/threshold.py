"""Adaptation of the feasibility threshold Delta (Algorithm 1, Sec. 4.7).

Start: Delta = 0.5, c = 0, step upsilon = 0.05.  After a batch of k evaluated
suggestions:
* some result invalid -> Delta = min(0.75, max(0.5, Delta + upsilon)), c = 0;
* otherwise           -> c = c + k; if c >= 5: Delta = max(0.25, Delta - upsilon), c = c - 5.
"""

DELTA0 = 0.5
UPSILON = 0.05


def delta_update(delta, c, k, any_invalid, upsilon=UPSILON):
    if any_invalid:
        return min(0.75, max(0.5, delta + upsilon)), 0
    c = c + k
    if c >= 5:
        delta = max(0.25, delta - upsilon)
        c = c - 5
    return delta, c
