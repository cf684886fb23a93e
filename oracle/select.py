"""Top-k parallel suggestion (Sec. 4.6): the k feasible candidates with the
largest acquisition value.

A candidate is eligible when its mask entry is non-zero and its score is not
NaN.  Order: score descending, then candidate index ascending (the lowest index
wins a tie).  Fewer than q eligible candidates leave -1 in the tail of the
index list; the paper fills such a shortfall with Sobol points (Sec. 4.7), a
step left to the caller.
"""
import numpy as np


def top_q(score, mask, q):
    """Returns (idx int64 (q,), score float64 (q,), n_valid)."""
    score = np.asarray(score, dtype=np.float64)
    idx_all = np.arange(len(score))
    ok = (np.asarray(mask) != 0) & ~np.isnan(score)
    cand = idx_all[ok]
    order = np.lexsort((cand, -score[cand]))
    pick = cand[order[:q]]
    idx = np.full(q, -1, dtype=np.int64)
    val = np.full(q, np.nan)
    idx[:len(pick)] = pick
    val[:len(pick)] = score[pick]
    return idx, val, int(ok.sum())
