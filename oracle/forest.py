"""Random-forest probability of feasibility and the hidden-constraint mask:
Sec. 4.7 and Eq. 3 (POF(x) >= Delta).

A forest is given as flat arrays (tree t owns nodes tree_offset[t] ..
tree_offset[t+1]-1; ``left``/``right`` are tree-local indices, -1 at a leaf):

* a walk starts at the tree's first node and goes left iff x[feature] <= threshold,
  the comparison taken in float32 (x and threshold are float32);
* each leaf holds its regression value v in Q16 fixed point, q = round(v * 2^16);
* votes(x) = sum over trees of q at the leaf reached, an exact integer;
* POF(x) = votes / (2^16 T), the mean of the trees' predictions;
* mask(x) = POF(x) >= Delta, decided on integers as votes >= ceil(Delta * (T * 2^16)),
  the threshold computed once in double precision.
"""
import math

import numpy as np


def forest_apply(forest, Xc):
    """Leaf reached in every tree, as tree-local node indices: (n, T) int32."""
    Xc = np.asarray(Xc, dtype=np.float32)
    feat, thr = forest["feature"], forest["threshold"].astype(np.float32)
    left, right, off = forest["left"], forest["right"], forest["tree_offset"]
    T = len(off) - 1
    n = len(Xc)
    leaves = np.empty((n, T), dtype=np.int32)
    rows = np.arange(n)
    for t in range(T):
        base = off[t]
        node = np.zeros(n, dtype=np.int64)
        while True:
            internal = left[base + node] >= 0
            if not internal.any():
                break
            g = base + node[internal]
            go_left = Xc[rows[internal], feat[g]] <= thr[g]
            node[internal] = np.where(go_left, left[g], right[g])
        leaves[:, t] = node
    return leaves


def forest_votes(forest, Xc):
    """Sum over trees of the Q16 leaf values: (n,) int64."""
    leaves = forest_apply(forest, Xc)
    off = forest["tree_offset"]
    q = forest["leaf_q16"].astype(np.int64)
    votes = np.zeros(len(leaves), dtype=np.int64)
    for t in range(leaves.shape[1]):
        votes += q[off[t] + leaves[:, t]]
    return votes


def vote_threshold(delta, n_trees):
    """Smallest integer vote count with POF >= Delta."""
    return int(math.ceil(float(delta) * float(n_trees * 65536)))


def feasibility_mask(votes, delta, n_trees):
    return (np.asarray(votes) >= vote_threshold(delta, n_trees)).astype(np.uint8)


def probability_of_feasibility(votes, n_trees):
    return np.asarray(votes, dtype=np.float64) / (65536.0 * n_trees)
