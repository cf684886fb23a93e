"""Pins of the forest mask (Sec. 4.7, Eq. 3), top-k (Sec. 4.6) and the
threshold adaptation (Algorithm 1)."""
import json
import os

import numpy as np
import pytest
from sklearn.ensemble import RandomForestRegressor

from oracle.forest import feasibility_mask, forest_apply, forest_votes, vote_threshold
from oracle.select import top_q
from oracle.threshold import delta_update
from workloads.synth import export_forest


def _hand(golden_dir):
    with open(os.path.join(golden_dir, "hand_trees.json")) as fh:
        g = json.load(fh)
    forest = {k: np.array(g[k]) for k in ("feature", "left", "right", "leaf_q16", "tree_offset")}
    forest["threshold"] = np.array(g["threshold"], dtype=np.float32)
    return g, forest


def test_hand_traced_trees(golden_dir):
    g, forest = _hand(golden_dir)
    X = np.array(g["X"], dtype=np.float32)
    assert forest_apply(forest, X).tolist() == g["leaves"]
    votes = forest_votes(forest, X)
    assert votes.tolist() == g["votes"]
    assert feasibility_mask(votes, 0.5, 3).tolist() == g["mask_delta_0.5"]
    assert feasibility_mask(votes, 0.6, 3).tolist() == g["mask_delta_0.6"]


def test_matches_sklearn_forest():
    rng = np.random.default_rng(21)
    X = rng.random((400, 6))
    y = ((X[:, 0] + X[:, 2] < 1.0) | (X[:, 4] > 0.8)).astype(float)
    model = RandomForestRegressor(n_estimators=12, max_depth=7, random_state=3).fit(X, y)
    forest = export_forest(model)
    Xc = rng.random((3000, 6)).astype(np.float32)
    Xc[:50, 0] = forest["threshold"][forest["feature"] == 0][:1]  # exact ties on a threshold
    leaves = forest_apply(forest, Xc)
    np.testing.assert_array_equal(leaves, model.apply(Xc))
    votes = forest_votes(forest, Xc)
    assert np.max(np.abs(votes / (65536.0 * 12) - model.predict(Xc))) <= 0.5 / 65536 + 1e-15


def test_vote_threshold():
    assert vote_threshold(0.5, 64) == 2097152
    assert vote_threshold(0.55, 64) == 2306868
    assert vote_threshold(0.25, 3) == 49152


def test_delta_sequences(golden_dir):
    with open(os.path.join(golden_dir, "delta_sequences.json")) as fh:
        g = json.load(fh)
    for seq in g["sequences"]:
        delta, c = 0.5, 0
        for k, bad, want_delta, want_c in seq["steps"]:
            delta, c = delta_update(delta, c, k, bad)
            assert delta == pytest.approx(want_delta, abs=1e-12)
            assert c == want_c


def _top_q_brute(score, mask, q):
    items = [(-s, i) for i, (s, m) in enumerate(zip(score, mask)) if m and not np.isnan(s)]
    items.sort()
    idx = [i for _, i in items[:q]] + [-1] * max(0, q - len(items))
    return idx, len(items)


def test_top_q_brute_force_and_ties():
    rng = np.random.default_rng(22)
    for _ in range(30):
        n = int(rng.integers(1, 60))
        score = rng.integers(0, 5, n).astype(float)
        score[rng.random(n) < 0.1] = np.nan
        mask = (rng.random(n) < 0.7).astype(np.uint8)
        q = int(rng.integers(1, 8))
        idx, val, nv = top_q(score, mask, q)
        want, wnv = _top_q_brute(score, mask, q)
        assert idx.tolist() == want and nv == wnv
    idx, _, nv = top_q(np.array([1.0, 3.0, 3.0, 2.0]), np.array([1, 1, 1, 1]), 2)
    assert idx.tolist() == [1, 2] and nv == 4
    idx, _, nv = top_q(np.array([1.0, 3.0]), np.array([0, 0]), 3)
    assert idx.tolist() == [-1, -1, -1] and nv == 0
