"""Pins of the forest-training oracle (Sec. 4.7) to scikit-learn's regression
trees (the paper's tool) and to the bootstrap's sampling law."""
import numpy as np
import pytest
from sklearn.tree import DecisionTreeRegressor

from oracle.forest_train import bootstrap_weights, predict, train_forest, train_tree


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
