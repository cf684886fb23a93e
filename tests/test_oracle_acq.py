"""Pins of EI (Eq. 8) and EHVI / hypervolume (Eq. 9, Sec. 4.4.2)."""
import itertools
import json
import os

import numpy as np
import pytest

from oracle.acquisition import expected_improvement, partial_expectation
from oracle.hypervolume import (column_boxes, ehvi, hvi_from_boxes, hypervolume,
                                hypervolume_2d_rectangles, hypervolume_improvement,
                                nondominated, nondominated_cells)


@pytest.fixture(scope="module")
def textbook(golden_dir):
    with open(os.path.join(golden_dir, "textbook_values.json")) as fh:
        return json.load(fh)


def test_partial_expectation_table(textbook):
    for case in textbook["partial_expectation"]:
        got = partial_expectation(case["c"], case["mu"], case["sigma"])
        assert float(got) == pytest.approx(case["G"], rel=1e-14, abs=1e-15)


def test_ei_monte_carlo():
    rng = np.random.default_rng(11)
    for mu, sd, best in [(0.3, 0.8, 0.1), (-1.0, 0.2, -0.9), (2.0, 1.5, 0.0)]:
        y = mu + sd * rng.standard_normal(1_000_000)
        imp = np.maximum(0.0, best + 1e-4 - y)
        se = imp.std() / np.sqrt(len(imp))
        assert abs(float(expected_improvement(mu, sd, best)) - imp.mean()) <= 5 * se + 1e-12


def test_ei_monte_carlo_with_xi():
    # a margin as large as the spread, so that its sign shows (the paper adds
    # xi to the improvement, Eq. 8; at xi = 1e-4 the test above cannot tell)
    rng = np.random.default_rng(12)
    for mu, sd, best, xi in [(0.3, 0.8, 0.1, 0.5), (-1.0, 0.2, -0.9, 0.1)]:
        y = mu + sd * rng.standard_normal(1_000_000)
        imp = np.maximum(0.0, best + xi - y)
        se = imp.std() / np.sqrt(len(imp))
        assert abs(float(expected_improvement(mu, sd, best, xi=xi)) - imp.mean()) <= 5 * se + 1e-12


def test_ei_jensen_and_monotone_in_sigma():
    mu = np.linspace(-2, 2, 41)
    for sd in [0.01, 0.3, 1.0]:
        ei = expected_improvement(mu, sd, 0.0, xi=0.0)
        assert np.all(ei >= np.maximum(0.0, -mu) - 1e-15)
    sds = np.linspace(0.01, 3.0, 50)
    ei = expected_improvement(0.5, sds, 0.0)
    assert np.all(np.diff(ei) > 0)


def test_hypervolume_hand_values(textbook):
    for case in textbook["hypervolume_2d"]:
        assert hypervolume(case["front"], np.array(case["ref"], float)) == pytest.approx(case["hv"], abs=1e-12)
        assert hypervolume_2d_rectangles(np.array(case["front"], float), np.array(case["ref"], float)) == \
            pytest.approx(case["hv"], abs=1e-12)
    for case in textbook["hypervolume_3d"]:
        assert hypervolume(case["front"], np.array(case["ref"], float)) == pytest.approx(case["hv"], abs=1e-12)


def _hv_inclusion_exclusion(P, ref):
    total = 0.0
    for k in range(1, len(P) + 1):
        for sub in itertools.combinations(range(len(P)), k):
            corner = np.max(P[list(sub)], axis=0)
            total += (-1) ** (k + 1) * np.prod(np.maximum(ref - corner, 0.0))
    return total


def test_hypervolume_inclusion_exclusion_and_mc():
    rng = np.random.default_rng(12)
    for p in (2, 3):
        for _ in range(5):
            P = rng.random((4, p))
            ref = np.ones(p) * 1.1
            hv = hypervolume(P, ref)
            assert hv == pytest.approx(_hv_inclusion_exclusion(P, ref), abs=1e-12)
            Z = rng.random((400_000, p)) * ref
            dom = np.zeros(len(Z), bool)
            for q in P:
                dom |= np.all(Z >= q, axis=1)
            frac = dom.mean()
            se = np.sqrt(frac * (1 - frac) / len(Z)) * np.prod(ref)
            assert abs(hv - frac * np.prod(ref)) <= 5 * se


def test_nondominated_filter():
    Y = np.array([[1, 3], [2, 2], [3, 1], [2.5, 2.5], [2, 2], [5, 0.5], [0.5, 5]], float)
    P = nondominated(Y, np.array([4.0, 4.0]))
    assert P.tolist() == [[1, 3], [2, 2], [3, 1]]


def test_hvi_from_boxes_matches_definition():
    rng = np.random.default_rng(13)
    for p in (2, 3):
        P = nondominated(rng.random((6, p)), np.ones(p))
        ref = np.ones(p) * 1.05
        for build in (nondominated_cells, column_boxes):
            lo, hi = build(P, ref)
            for _ in range(20):
                y = rng.random(p) * 1.2 - 0.1
                assert hvi_from_boxes(y, lo, hi) == pytest.approx(hypervolume_improvement(y, P, ref), abs=1e-12)


def test_ehvi_monte_carlo():
    rng = np.random.default_rng(14)
    for p, size in ((2, 5), (3, 4)):
        P = nondominated(rng.random((size, p)), np.ones(p))
        ref = np.ones(p) * 1.1
        mu = rng.random(p)
        sd = rng.uniform(0.05, 0.4, p)
        lo, hi = column_boxes(P, ref)
        Ys = mu + sd * rng.standard_normal((200_000, p))
        vals = np.array([hvi_from_boxes(y, lo, hi) for y in Ys])
        se = vals.std() / np.sqrt(len(vals))
        got = ehvi(mu[None, :], sd[None, :], P, ref)[0]
        assert abs(got - vals.mean()) <= 5 * se


def test_ehvi_limits_and_invariances():
    rng = np.random.default_rng(15)
    P = nondominated(rng.random((6, 2)), np.ones(2))
    ref = np.array([1.1, 1.2])
    mu = rng.random((30, 2))
    # sigma -> 0 gives HVI(mu)
    got = ehvi(mu, np.zeros_like(mu), P, ref)
    want = [hypervolume_improvement(m, P, ref) for m in mu]
    np.testing.assert_allclose(got, want, atol=1e-12)
    sd = rng.uniform(0.05, 0.5, mu.shape)
    e = ehvi(mu, sd, P, ref)
    assert np.all(e >= 0)
    # empty front: product of G_j(r_j)
    e0 = ehvi(mu, sd, np.zeros((0, 2)), ref)
    np.testing.assert_allclose(e0, partial_expectation(ref[0], mu[:, 0], sd[:, 0]) *
                               partial_expectation(ref[1], mu[:, 1], sd[:, 1]), rtol=1e-13)
    # a dominated extra point changes nothing; permuting objectives changes nothing
    P_dom = np.vstack([P, P[0] + 0.01])
    np.testing.assert_allclose(ehvi(mu, sd, nondominated(P_dom, ref), ref), e, rtol=1e-13)
    np.testing.assert_allclose(ehvi(mu[:, ::-1], sd[:, ::-1], P[:, ::-1], ref[::-1]), e, rtol=1e-12)
    # the full grid and the merged columns agree
    np.testing.assert_allclose(ehvi(mu, sd, P, ref, boxes="cells"), e, rtol=1e-12, atol=1e-15)
    P3 = nondominated(rng.random((7, 3)), np.ones(3))
    mu3, sd3 = rng.random((10, 3)), rng.uniform(0.05, 0.5, (10, 3))
    np.testing.assert_allclose(ehvi(mu3, sd3, P3, np.ones(3)), ehvi(mu3, sd3, P3, np.ones(3), boxes="cells"),
                               rtol=1e-12, atol=1e-15)


def test_ehvi_one_objective_is_ei():
    mu = np.linspace(-1, 1, 9)[:, None]
    sd = np.full_like(mu, 0.3)
    best = -0.2
    got = ehvi(mu, sd, np.array([[best]]), np.array([5.0]))
    np.testing.assert_allclose(got, expected_improvement(mu[:, 0], sd[:, 0], best, xi=0.0), rtol=1e-13)
