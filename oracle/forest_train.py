"""Training the feasibility forest (Sec. 4.7: a random forest regressor on
the evaluated configurations, label 1 = the engine ran, 0 = it crashed).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Each tree is a regression tree grown by exhaustive search (CART): a node
holding samples S (with bootstrap multiplicities w) is split on the feature
and threshold that maximise the decrease of the weighted sum of squared
deviations of the labels, which is the same as maximising

    proxy = sum_L^2 / w_L + sum_R^2 / w_R

(sum_L, w_L: weighted label sum and weight left of the threshold).  The
features are first rounded to float32 (the candidates the forest judges are
float32).  Thresholds are midpoints a/2 + b/2 between consecutive distinct
feature values a < b (a itself if that rounds up to b); equal proxies go to
the lower feature index, then the lower threshold.  A node becomes a leaf
(value: the weighted mean label) at max_depth, with fewer than 2 samples, when
its labels are all equal, or when no split decreases the squared deviation.

Forest: tree t is grown on a bootstrap sample of the N draws: draw j (j = 0 ..
N-1) picks sample floor(u * N), u the top 53 bits of output t * N + j of
SplitMix64 started from ``seed`` (see ``mace``) over 2^53; with
bootstrap=False every tree sees every draw once.  All features are candidates
at every split (max_features = d).
"""
import numpy as np

from .mace import splitmix64


def _grow(X, y, w, idx, depth, max_depth, nodes):
    """Appends the subtree over samples idx (preorder, left first); returns its node index."""
    me = len(nodes)
    wy = w[idx] * y[idx]
    W = w[idx].sum()
    nodes.append(dict(feature=-1, threshold=0.0, left=-1, right=-1, value=wy.sum() / W))
    if depth >= max_depth or len(idx) < 2 or np.all(y[idx] == y[idx][0]):
        return me
    total = wy.sum()
    best = (total * total / W, -1, 0.0)  # a split must beat the unsplit node
    for f in range(X.shape[1]):
        order = idx[np.argsort(X[idx, f], kind="stable")]
        xs = X[order, f]
        sl = wl = 0.0
        for p in range(len(order) - 1):
            sl += w[order[p]] * y[order[p]]
            wl += w[order[p]]
            if xs[p + 1] == xs[p]:
                continue
            sr, wr = total - sl, W - wl
            proxy = sl * sl / wl + sr * sr / wr
            if proxy > best[0]:
                t = xs[p] / 2.0 + xs[p + 1] / 2.0
                best = (proxy, f, xs[p] if t == xs[p + 1] else t)
    if best[1] < 0:
        return me
    f, t = best[1], best[2]
    go_left = X[idx, f] <= t
    nodes[me]["feature"], nodes[me]["threshold"] = f, t
    nodes[me]["left"] = _grow(X, y, w, idx[go_left], depth + 1, max_depth, nodes)
    nodes[me]["right"] = _grow(X, y, w, idx[~go_left], depth + 1, max_depth, nodes)
    return me


def train_tree(X, y, max_depth, weights=None):
    """One regression tree; returns a list of node dicts in preorder."""
    X = np.asarray(X, dtype=np.float32).astype(np.float64)
    y = np.asarray(y, dtype=np.float64)
    w = np.ones(len(X)) if weights is None else np.asarray(weights, dtype=np.float64)
    idx = np.flatnonzero(w > 0)
    nodes = []
    _grow(X, y, w, idx, 0, max_depth, nodes)
    return nodes


def bootstrap_weights(n, tree, seed):
    """Multiplicity of every draw in tree ``tree``'s bootstrap sample."""
    w = np.zeros(n)
    for j in range(n):
        u = (splitmix64(seed, tree * n + j) >> 11) / float(1 << 53)
        w[int(u * n)] += 1
    return w


def train_forest(X, y, n_trees, max_depth, seed, bootstrap=True):
    """Flat arrays as the forest loader takes them: feature, threshold
    (float64), left, right, value, tree_offset."""
    n = len(X)
    feature, threshold, left, right, value, offset = [], [], [], [], [], [0]
    for t in range(n_trees):
        w = bootstrap_weights(n, t, seed) if bootstrap else None
        nodes = train_tree(X, y, max_depth, w)
        for nd in nodes:
            feature.append(nd["feature"] if nd["left"] >= 0 else -1)
            threshold.append(nd["threshold"])
            left.append(nd["left"])
            right.append(nd["right"])
            value.append(nd["value"])
        offset.append(offset[-1] + len(nodes))
    return dict(feature=np.array(feature, np.int32), threshold=np.array(threshold), left=np.array(left, np.int32),
                right=np.array(right, np.int32), value=np.array(value), tree_offset=np.array(offset, np.int64))


def predict(forest, X):
    """Mean over trees of the reached leaf values (float64)."""
    X = np.asarray(X, dtype=np.float64)
    out = np.zeros(len(X))
    T = len(forest["tree_offset"]) - 1
    for t in range(T):
        base = forest["tree_offset"][t]
        for i, x in enumerate(X):
            k = 0
            while forest["left"][base + k] >= 0:
                k = forest["left"][base + k] if x[forest["feature"][base + k]] <= forest["threshold"][base + k] \
                    else forest["right"][base + k]
            out[i] += forest["value"][base + k]
    return out / T


def voting_format(tf):
    """A trained forest in the form the vote count of Eq. 3 reads (float32
    compares, integer Q16 votes): each float64 threshold t becomes the largest float32 not
    above t, so a float32 feature x goes left exactly when x <= t; each leaf
    value v becomes round(v * 2^16), ties to even."""
    t64 = np.asarray(tf["threshold"], dtype=np.float64)
    t32 = t64.astype(np.float32)
    above = t32.astype(np.float64) > t64
    t32[above] = np.nextafter(t32[above], np.float32(-np.inf))
    leaf = np.asarray(tf["left"]) < 0
    return dict(feature=np.where(leaf, 0, tf["feature"]).astype(np.int32),
                threshold=np.where(leaf, np.float32(0), t32).astype(np.float32),
                left=np.asarray(tf["left"], np.int32), right=np.asarray(tf["right"], np.int32),
                leaf_q16=np.where(leaf, np.rint(np.asarray(tf["value"]) * 65536.0), 0).astype(np.int32),
                tree_offset=np.asarray(tf["tree_offset"], np.int64))
