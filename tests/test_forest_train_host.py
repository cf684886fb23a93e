"""The library's forest training (host; Sec. 4.7) against the oracle: the
same trees node for node on the same draws and seed.  No device work."""
import time

import numpy as np
import pytest

import paper_2408_04323_amd as S
from oracle.forest_train import train_forest
from workloads import make_workload


def _same(a, b):
    for k in ("feature", "left", "right", "tree_offset"):
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)
    np.testing.assert_array_equal(a["threshold"], b["threshold"])
    np.testing.assert_array_equal(a["value"], b["value"])


@pytest.mark.parametrize("n,d,T,depth,boot", [(60, 3, 4, 5, True), (300, 8, 6, 10, True), (200, 5, 2, 64, False),
                                              (1, 2, 2, 3, True), (50, 4, 3, 0, True)])
def test_forest_matches_oracle(n, d, T, depth, boot):
    rng = np.random.default_rng(n + d)
    X = rng.random((n, d))
    X[:, -1] = np.round(X[:, -1] * 3) / 3  # a grid dimension: ties in the features
    y = ((X[:, 0] + 0.3 * X[:, 1] + 0.2 * rng.standard_normal(n)) < 0.8).astype(float)
    got = S.forest_train(X, y, T, depth, seed=777, bootstrap=boot)
    want = train_forest(X, y, T, depth, seed=777, bootstrap=boot)
    _same(got, want)


def test_workload_draws_match_oracle_and_time():
    """The two-objective workload's draws (every evaluated configuration with its crash label)."""
    w = make_workload(3, n=16, with_forest=False)
    X, y = w["X_draws"], w["feasible_draws"]
    t0 = time.perf_counter()
    got = S.forest_train(X, y, 64, 10, seed=240804323)
    el = time.perf_counter() - t0
    print(f"[forest train] {len(X)} draws, d={X.shape[1]}, 64 trees depth 10: {len(got['feature'])} nodes, {el:.3f} s")
    want = train_forest(X, y, 8, 10, seed=240804323)  # the oracle is slow: compare the first eight trees
    k = want["tree_offset"][-1]
    for key in ("feature", "left", "right", "threshold", "value"):
        np.testing.assert_array_equal(got[key][:k], want[key], err_msg=key)


def test_errors():
    X = np.zeros((3, 2))
    with pytest.raises(S.ScootError):
        S.forest_train(X, np.array([0.0, 1.0, np.nan]), 2, 3, 0)
    with pytest.raises(S.ScootError):
        S.forest_train(np.zeros((3, 17)), np.zeros(3), 2, 3, 0)
