"""Pins of the candidate-generation oracle: scipy's Sobol generator (an
independent implementation, with the direction-number table it ships),
hand-worked first points, the net property, grids and known constraints."""
import glob
import os

import numpy as np
import pytest
import scipy
from scipy.stats import qmc

from oracle.sobol import direction_numbers, known_constraints_mask, snap_levels, sobol_points, sobol_pool


def _table(d):
    f = glob.glob(os.path.join(os.path.dirname(scipy.__file__), "stats", "_sobol_direction_numbers.npz"))[0]
    z = np.load(f, allow_pickle=False)
    return z["poly"][:d].astype(np.int64), z["vinit"][:d].astype(np.int64)


@pytest.mark.parametrize("d,n", [(1, 64), (5, 1024), (16, 4096)])
def test_points_match_scipy(d, n):
    poly, vinit = _table(d)
    want = qmc.Sobol(d, scramble=False).random(n)
    np.testing.assert_array_equal(sobol_points(poly, vinit, n), want)


def test_skip_continues_the_sequence():
    poly, vinit = _table(4)
    np.testing.assert_array_equal(sobol_points(poly, vinit, 40, skip=100), sobol_points(poly, vinit, 140)[100:])


def test_first_points_by_hand():
    # dimension 0: van der Corput in Gray-code order 0, 1/2, 3/4, 1/4, 3/8, 7/8, 5/8, 1/8
    # dimension 1: x + 1, m_1 = 1: V = 1/2, 3/4 (m_2 = 2 m_1 ^ m_1 = 3), ...
    poly, vinit = _table(2)
    P = sobol_points(poly, vinit, 8)
    np.testing.assert_array_equal(P[:, 0], [0, .5, .75, .25, .375, .875, .625, .125])
    np.testing.assert_array_equal(P[:4, 1], [0, .5, .25, .75])
    assert direction_numbers(3, [1])[:3] == [1 << 31, 3 << 30, 5 << 29]


def test_net_property():
    poly, vinit = _table(6)
    P = sobol_points(poly, vinit, 256)
    for j in range(6):  # each one-dimensional projection of the first 2^k points is {i / 2^k}
        np.testing.assert_array_equal(np.sort(P[:256, j]), np.arange(256) / 256)


def test_grids_and_booleans():
    U = np.array([[0.5, 0.5, 0.5, 0.49], [0.1, 0.74, 0.2, 0.51]])
    X = snap_levels(U, [0, 1, 3, 5])
    np.testing.assert_array_equal(X[:, 0], [0.5, 0.1])
    np.testing.assert_array_equal(X[:, 1], [1.0, 1.0])            # boolean: x >= 1/2
    np.testing.assert_array_equal(X[:, 2], [0.5, 0.0])            # 3 levels {0, 1/2, 1}
    np.testing.assert_array_equal(X[:, 3], [0.5, 0.5])            # 5 levels, 0.49 * 4 = 1.96 -> 2
    poly, vinit = _table(3)
    pool = sobol_pool(poly, vinit, [0, 1, 9], 100)
    assert pool.dtype == np.float32 and set(np.unique(pool[:, 1])) <= {0.0, 1.0}
    assert np.all(np.isin(np.round(pool[:, 2] * 8, 6), np.arange(9)))


def test_known_constraints():
    X = np.array([[0.2, 0.3], [0.6, 0.6], [0.5, 0.5]], dtype=np.float32)
    A = np.array([[1.0, 1.0], [-1.0, 0.0]])
    b = np.array([1.0, -0.1])      # x0 + x1 <= 1 and x0 >= 0.1
    np.testing.assert_array_equal(known_constraints_mask(X, A, b), [1, 0, 1])   # 0.5 + 0.5 <= 1 holds
    assert known_constraints_mask(X, np.zeros((0, 2)), np.zeros(0)).tolist() == [1, 1, 1]


def test_known_constraints_encode_the_engine_rules():
    """The linear rows of the vLLM-like space decide exactly what the engine's
    rules, checked in engine units, decide -- on a Sobol pool of the space,
    where the integer knobs meet their boundaries (equal token and sequence
    limits, tokens exactly at the model length) many times."""
    from workloads import sobol_table, vllm_decode, vllm_space
    sp = vllm_space()
    poly, vinit = sobol_table(sp["d"])
    X = sobol_pool(poly, vinit, sp["levels"], 4096)
    # add hand-made boundary rows: tokens == seqs, tokens == 4096 without chunking, both booleans
    span = 8128.0
    extra = np.array(X[:6], dtype=np.float64)
    extra[0, 1] = extra[0, 2] = (4096 - 64) / span
    extra[0, 5] = extra[0, 6] = 0.0
    extra[1, 1], extra[1, 2] = (1000 - 64) / span, (999 - 64) / span
    extra[2, 2], extra[2, 5], extra[2, 6] = (4095 - 64) / span, 0.0, 0.0
    extra[3, 2], extra[3, 1], extra[3, 5], extra[3, 6] = (4095 - 64) / span, 0.0, 1.0, 0.0
    extra[4, 5] = extra[4, 6] = 1.0
    extra[5, 1], extra[5, 2], extra[5, 5], extra[5, 6] = 0.0, 1.0, 1.0, 0.0
    X = np.vstack([X, extra.astype(np.float32)])
    got = known_constraints_mask(X, sp["A"], sp["b"])
    v = vllm_decode(X.astype(np.float64))
    tok, seqs = v["max-num-batched-tokens"], v["max-num-seqs"]
    chunk, prefix = v["enable-chunked-prefill"], v["enable-prefix-caching"]
    want = (tok >= seqs) & ~(chunk & prefix) & (chunk | (tok >= 4096))
    np.testing.assert_array_equal(got, want.astype(np.uint8))
    assert list(got[-6:]) == [1, 0, 0, 1, 0, 1]
    assert np.sum(tok == seqs) > 0 and 0.2 < got.mean() < 0.8
