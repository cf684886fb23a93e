"""Pins of the forest-training oracle (Sec. 4.7) to scikit-learn's regression
trees (the paper's tool) and to the bootstrap's sampling law."""
import numpy as np
import pytest
from sklearn.tree import DecisionTreeRegressor

from oracle.forest_train import bootstrap_weights, predict, train_forest, train_tree, voting_format


def _sk_nodes(model):
    t = model.tree_
    return [dict(feature=int(t.feature[k]) if t.children_left[k] >= 0 else -1,
                 threshold=float(t.threshold[k]) if t.children_left[k] >= 0 else 0.0,
                 left=int(t.children_left[k]), right=int(t.children_right[k]), value=float(t.value[k].ravel()[0]))
            for k in range(t.node_count)]


def _membership(nodes, X):
    """Which nodes each sample passes through, walking the oracle's tree."""
    M = np.zeros((len(X), len(nodes)), dtype=bool)
    for i, x in enumerate(np.asarray(X, np.float32).astype(np.float64)):
        k = 0
        M[i, 0] = True
        while nodes[k]["left"] >= 0:
            k = nodes[k]["left"] if x[nodes[k]["feature"]] <= nodes[k]["threshold"] else nodes[k]["right"]
            M[i, k] = True
    return M


@pytest.mark.parametrize("seed,depth", [(0, 3), (1, 6), (2, 12)])
def test_single_tree_matches_sklearn(seed, depth):
    """Continuous features and targets: the exhaustive CART tree is sklearn's
    up to exact ties.  Two features can order a small node's samples the same
    way (or mirrored) and tie exactly; sklearn breaks such ties by its random
    feature order, the oracle by the lower index, so the comparison is of
    partitions: every node splits its training samples into the same two
    sets (in either order), leaves carry the same values, and where both
    chose the same feature the thresholds are equal."""
    rng = np.random.default_rng(seed)
    X = rng.random((150, 4)).astype(np.float32).astype(np.float64)
    y = np.sin(5 * X[:, 0]) + X[:, 1] * X[:, 2] + 0.1 * rng.standard_normal(150)
    sk = DecisionTreeRegressor(max_depth=depth, random_state=0).fit(X, y)
    mine = train_tree(X, y, depth)
    ref = _sk_nodes(sk)
    A = _membership(mine, X)
    B = sk.decision_path(X).toarray().astype(bool)
    assert len(mine) == len(ref)

    def same(k, j):
        assert np.array_equal(A[:, k], B[:, j])
        a, b = mine[k], ref[j]
        assert a["value"] == pytest.approx(b["value"], rel=1e-12, abs=1e-12)
        assert (a["left"] < 0) == (b["left"] < 0)
        if a["left"] < 0:
            return
        if a["feature"] == b["feature"]:
            assert a["threshold"] == b["threshold"]
        if np.array_equal(A[:, a["left"]], B[:, b["left"]]):
            same(a["left"], b["left"])
            same(a["right"], b["right"])
        else:
            same(a["left"], b["right"])
            same(a["right"], b["left"])

    same(0, 0)


def test_weights_equal_repeated_rows():
    """A multiplicity is the same as repeating the row."""
    rng = np.random.default_rng(3)
    X = rng.random((40, 3))
    y = (X[:, 0] + 0.3 * rng.standard_normal(40) > 0.5).astype(float)
    w = rng.integers(0, 4, 40).astype(float)
    reps = np.repeat(np.arange(40), w.astype(int))
    a, b = train_tree(X, y, 6, w), train_tree(X[reps], y[reps], 6)
    assert [(n["feature"], n["threshold"], n["left"]) for n in a] == [(n["feature"], n["threshold"], n["left"])
                                                                       for n in b]
    np.testing.assert_allclose([n["value"] for n in a], [n["value"] for n in b], rtol=1e-12)


def test_leaves_fit_the_training_labels_at_full_depth():
    rng = np.random.default_rng(4)
    X = rng.random((80, 2))
    y = (X[:, 0] > X[:, 1]).astype(float)
    f = train_forest(X, y, 1, 30, seed=0, bootstrap=False)
    np.testing.assert_array_equal(predict(f, X), y)


def test_bootstrap_sampling_law():
    n, T = 500, 60
    W = np.array([bootstrap_weights(n, t, 12345) for t in range(T)])
    assert np.all(W.sum(axis=1) == n)
    # each draw appears Binomial(n, 1/n) times: about 1 - 1/e of the draws are in a sample
    frac = (W > 0).mean()
    assert frac == pytest.approx(1 - np.exp(-1), abs=0.01)
    assert W.mean() == pytest.approx(1.0) and W.var() == pytest.approx(1 - 1 / n, rel=0.05)
    assert not np.array_equal(W[0], W[1])


# ------------------------------------------------ the voting format (Eq. 3)
def _f32_neighbours(t):
    t = np.float32(t)
    return [np.nextafter(t, np.float32(-np.inf)), t, np.nextafter(t, np.float32(np.inf))]


def _one_split(threshold, left_value=0.0, right_value=1.0):
    return dict(feature=np.array([0, -1, -1], np.int32), threshold=np.array([threshold, 0.0, 0.0]),
                left=np.array([1, -1, -1], np.int32), right=np.array([2, -1, -1], np.int32),
                value=np.array([0.5, left_value, right_value]), tree_offset=np.array([0, 3], np.int64))


A32 = float(np.float32(0.3))                     # 0.3 rounded to float32, exactly
UP32 = float(np.nextafter(np.float32(0.3), np.float32(1)))
THRESHOLDS = [
    (A32, A32),                                  # already a float32: kept
    (A32 + 1e-12, A32),                          # just above a float32 (rounds to nearest A32): down to A32
    (A32 - 1e-12, float(np.nextafter(np.float32(A32), np.float32(0)))),   # just below: the float32 below
    (UP32 - 1e-12, A32),                         # just below the next float32 (nearest is UP32): A32
    (0.1, float(np.float32(0.1)) if float(np.float32(0.1)) <= 0.1 else
     float(np.nextafter(np.float32(0.1), np.float32(0)))),
]


@pytest.mark.parametrize("t64,want", THRESHOLDS)
def test_voting_format_threshold_is_the_float32_below(t64, want):
    """The float32 threshold is the largest float32 not above the float64 one,
    so every float32 feature goes the same way under both."""
    f = voting_format(_one_split(t64))
    t32 = f["threshold"][0]
    assert f["threshold"].dtype == np.float32
    assert float(t32) == want
    assert float(t32) <= t64 < float(np.nextafter(t32, np.float32(np.inf)))
    for x in _f32_neighbours(want) + _f32_neighbours(t64):
        assert (x <= t32) == (float(x) <= t64)


@pytest.mark.parametrize("value,q16", [
    (0.0, 0), (1.0, 65536), (0.5, 32768), (0.7, 45875),          # 0.7 * 2^16 = 45875.2
    (0.5 / 65536, 0), (1.5 / 65536, 2), (2.5 / 65536, 2), (3.5 / 65536, 4),   # exact half steps: to even
    (12345.5 / 65536, 12346), (12346.5 / 65536, 12346),
])
def test_voting_format_leaf_q16_ties_to_even(value, q16):
    f = voting_format(_one_split(0.5, left_value=value))
    assert f["leaf_q16"][1] == q16
    assert f["leaf_q16"][0] == 0 and f["leaf_q16"][2] == 65536 and f["feature"][1] == 0


def test_voting_format_votes_match_the_float64_walk():
    """Votes of a trained forest in the voting format, over float32 inputs that
    include every threshold and its float32 neighbours, equal the sum over
    trees of round(2^16 v), v the value the float64 walk of the trained trees
    reaches."""
    rng = np.random.default_rng(11)
    X = rng.random((300, 3)).astype(np.float32)
    y = ((X[:, 0] + X[:, 1] > 1.0) ^ (rng.random(300) < 0.1)).astype(float)
    tf = train_forest(X, y, 5, 7, seed=5)
    fmt = voting_format(tf)
    from oracle.forest import forest_votes
    probes = [X]
    for k in np.flatnonzero(tf["left"] >= 0):
        f = tf["feature"][k]
        for x in _f32_neighbours(tf["threshold"][k]):
            row = X[k % len(X)].copy()
            row[f] = x
            probes.append(row[None, :])
    P = np.vstack(probes).astype(np.float32)
    want = np.zeros(len(P), np.int64)
    for t in range(len(tf["tree_offset"]) - 1):
        base = tf["tree_offset"][t]
        for i, x in enumerate(P.astype(np.float64)):
            k = 0
            while tf["left"][base + k] >= 0:
                k = tf["left"][base + k] if x[tf["feature"][base + k]] <= tf["threshold"][base + k] \
                    else tf["right"][base + k]
            want[i] += int(np.rint(tf["value"][base + k] * 65536.0))
    np.testing.assert_array_equal(forest_votes(fmt, P), want)
    # and POF is the float64 prediction to within half a step per tree
    np.testing.assert_allclose(want / (65536.0 * 5), predict(tf, P), rtol=0, atol=0.5 / 65536)
