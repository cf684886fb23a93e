"""Pins of the MACE oracle (Sec. 4.5.1; Eq. 6-8; pick of Sec. 4.6) against
values and properties that do not come from the oracle itself."""
import math

import numpy as np
import pytest

from oracle.mace import (GOLDEN_GAMMA, MASK64, mace_scores, pareto_front_max, probability_of_improvement,
                         random_pick, splitmix64, splitmix64_mix, ucb_beta, ucb_score)


def test_ucb_beta_hand_values():
    # t = 1: delta = 1, beta = 2 ln(pi^2 / 6) = 2 ln(1.6449340668)
    #   = 2 (ln 1.64 + ln 1.0030085773) = 2 (0.4946962418 + 0.0030040607) = 0.9954006050
    assert ucb_beta(1) == pytest.approx(0.9954006050, rel=1e-9)
    # t = 2: delta = 1/4, beta = 2 ln(16 pi^2 / 6) = 0.9954006050 + 8 ln 2 = 6.5405780494
    assert ucb_beta(2) == pytest.approx(6.5405780494, rel=1e-9)
    # beta_t = 2 ln(pi^2 / 6) + 8 ln t
    for t in (3, 10, 100):
        assert ucb_beta(t) == pytest.approx(0.9954006050 + 8 * math.log(t), rel=1e-9)


def test_ucb_score_is_the_mirrored_eq6():
    mu = np.array([0.0, 1.0, -2.0])
    sd = np.array([1.0, 0.5, 0.0])
    # the paper maximises f = -y: mean of f is -mu, plus beta sigma
    np.testing.assert_array_equal(ucb_score(mu, sd, 2.0), np.array([2.0, 0.0, 2.0]))


def test_pi_textbook_values():
    # standard normal table: Phi(1) = 0.8413447461, Phi(-1.959964) = 0.0250000
    assert probability_of_improvement(np.array([0.0]), np.array([1.0]), 1.0, 0.0)[0] == \
        pytest.approx(0.8413447461, abs=1e-10)
    assert probability_of_improvement(np.array([1.959964]), np.array([1.0]), 0.0, 0.0)[0] == \
        pytest.approx(0.025, abs=1e-7)
    # at the threshold itself the probability is one half; xi moves the threshold up
    assert probability_of_improvement(np.array([0.3]), np.array([2.0]), 0.2, 0.1)[0] == pytest.approx(0.5)


def test_pi_monte_carlo():
    rng = np.random.default_rng(5)
    mu, sd, best, xi = 0.4, 0.7, 0.1, 1e-4
    y = rng.normal(mu, sd, 2_000_000)
    mc = np.mean(y < best + xi)
    assert probability_of_improvement(np.array([mu]), np.array([sd]), best, xi)[0] == pytest.approx(mc, abs=2e-3)


def test_pi_monte_carlo_with_xi():
    # a margin as large as the spread, so that its sign shows (Eq. 7 adds xi)
    rng = np.random.default_rng(6)
    mu, sd, best, xi = 0.4, 0.7, 0.1, 0.3
    y = rng.normal(mu, sd, 2_000_000)
    mc = np.mean(y < best + xi)
    assert probability_of_improvement(np.array([mu]), np.array([sd]), best, xi)[0] == pytest.approx(mc, abs=2e-3)


def test_pi_zero_sigma_is_a_step():
    got = probability_of_improvement(np.array([-1.0, 1.0, 0.5]), np.zeros(3), 0.5, 0.0)
    np.testing.assert_array_equal(got, [1.0, 0.0, 0.0])


def test_mace_scores_monotone_in_mean():
    mu = np.linspace(-2, 2, 50)
    sd = np.full(50, 0.6)
    ucb, pi, ei = mace_scores(mu, sd, 0.0, 1e-4, 1.5)
    for s in (ucb, pi, ei):
        assert np.all(np.diff(s) < 0)


# ---------------------------------------------------------------- Pareto front

def test_front_hand_example():
    # (ucb, pi, ei) for six candidates, worked by hand:
    #   0 = (3, 0.2, 1) front (best ucb)
    #   1 = (1, 0.9, 1) front (best pi)
    #   2 = (2, 0.5, 2) front (best ei)
    #   3 = (1, 0.5, 1) dominated by 1 (0.9 > 0.5) and by 2
    #   4 = (2, 0.5, 2) equal to 2: equal vectors do not dominate, front
    #   5 = (3, 0.2, 0.5) dominated by 0 (ei 1 > 0.5)
    S = np.array([[3, .2, 1], [1, .9, 1], [2, .5, 2], [1, .5, 1], [2, .5, 2], [3, .2, .5]])
    np.testing.assert_array_equal(pareto_front_max(S), [1, 1, 1, 0, 1, 0])
    # masking out 2 and 4 frees nothing else; masking out 0 frees 5
    np.testing.assert_array_equal(pareto_front_max(S, [1, 1, 0, 1, 0, 1]), [1, 1, 0, 0, 0, 0])
    np.testing.assert_array_equal(pareto_front_max(S, [0, 1, 1, 1, 1, 1]), [0, 1, 1, 0, 1, 1])


def _skyline_2d(a, b):
    """Independent 2-D maxima by a sweep: sort by a descending; a point is on
    the front iff its b is the largest of its a-group and exceeds every b of
    the strictly larger a's."""
    order = np.lexsort((-b, -a))
    out = np.zeros(len(a), dtype=bool)
    best_prev = -np.inf
    k = 0
    while k < len(order):
        j = k
        while j < len(order) and a[order[j]] == a[order[k]]:
            j += 1
        group = order[k:j]
        gmax = b[group].max()
        if gmax > best_prev:
            out[group[b[group] == gmax]] = True
        best_prev = max(best_prev, gmax)
        k = j
    return out


@pytest.mark.parametrize("seed", range(6))
def test_front_2d_matches_sweep(seed):
    rng = np.random.default_rng(seed)
    n = 300
    a = rng.integers(0, 12, n).astype(float)  # ties on purpose
    b = rng.integers(0, 12, n).astype(float)
    S = np.stack([a, b, np.zeros(n)], axis=1)
    np.testing.assert_array_equal(pareto_front_max(S), _skyline_2d(a, b))


def test_front_one_score_is_the_argmax_set():
    v = np.array([1.0, 3.0, 2.0, 3.0, -1.0])
    S = np.stack([v, v, v], axis=1)
    np.testing.assert_array_equal(pareto_front_max(S), v == 3.0)


@pytest.mark.parametrize("seed", range(4))
def test_front_invariants(seed):
    rng = np.random.default_rng(10 + seed)
    n = 400
    z = rng.standard_normal((n, 3))
    S = z @ np.array([[1, .6, .2], [0, .8, .3], [0, 0, .9]])
    S[rng.integers(0, n, 20)] = S[rng.integers(0, n, 20)]  # duplicates
    mask = rng.random(n) < 0.8
    f = pareto_front_max(S, mask)
    F = S[f]
    assert f.any() and not (f & ~mask).any()
    for i in np.flatnonzero(f):  # front members: nobody eligible dominates them
        assert not (((S[mask] >= S[i]).all(1)) & ((S[mask] > S[i]).any(1))).any()
    for i in np.flatnonzero(mask & ~f):  # the rest: some front member dominates each
        assert (((F >= S[i]).all(1)) & ((F > S[i]).any(1))).any()
    perm = rng.permutation(n)
    np.testing.assert_array_equal(pareto_front_max(S[perm], mask[perm]), f[perm])


def test_front_nan_is_ineligible():
    S = np.array([[1.0, 1.0, 1.0], [np.nan, 5.0, 5.0], [0.5, 0.5, 0.5]])
    np.testing.assert_array_equal(pareto_front_max(S), [True, False, False])


# ------------------------------------------------------------ the random pick

def test_golden_gamma_is_the_odd_integer_nearest_2_64_over_phi():
    # 2^64 / phi = 2^63 (sqrt 5 - 1); floor via an exact integer square root
    floor_val = math.isqrt(5 << 126) - (1 << 63)
    assert GOLDEN_GAMMA in (floor_val, floor_val + 1) and GOLDEN_GAMMA % 2 == 1


def test_splitmix_reference_outputs():
    # the published first outputs of SplitMix64 seeded with 0
    assert [splitmix64(0, i) for i in range(3)] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_splitmix_stream_and_bijection():
    seed = 0x1234_5678_9ABC_DEF0
    for i in range(5):
        assert splitmix64(seed, i) == splitmix64_mix((seed + (i + 1) * GOLDEN_GAMMA) & MASK64)
    outs = {splitmix64(seed, i) for i in range(20000)}
    assert len(outs) == 20000


def test_splitmix_avalanche():
    """Each input bit flips each output bit about half the time: a dropped
    xor-shift or a wrong shift amount fails this."""
    rng = np.random.default_rng(7)
    xs = [int(v) for v in rng.integers(0, 2 ** 63, 400, dtype=np.int64)]
    flips = np.zeros((64, 64))
    for x in xs:
        y = splitmix64_mix(x)
        for b in range(64):
            d = y ^ splitmix64_mix(x ^ (1 << b))
            flips[b] += [(d >> k) & 1 for k in range(64)]
    frac = flips / len(xs)
    assert np.all(np.abs(frac - 0.5) < 0.12)
    assert abs(frac.mean() - 0.5) < 0.01


def test_random_pick_is_uniform_over_subsets():
    flags = np.zeros(50, dtype=np.uint8)
    members = [3, 11, 17, 29, 40, 44]
    flags[members] = 1
    counts = {}
    trials = 6000
    for seed in range(trials):
        idx, nf = random_pick(flags, seed, 2)
        assert nf == 6 and set(idx) <= set(members) and idx[0] != idx[1]
        key = tuple(sorted(idx))
        counts[key] = counts.get(key, 0) + 1
    assert len(counts) == 15
    expected = trials / 15
    chi2 = sum((c - expected) ** 2 / expected for c in counts.values())
    assert chi2 < 36.1  # 99.9% quantile of chi-square with 14 degrees of freedom


def test_random_pick_shortfall_and_determinism():
    flags = np.zeros(10, dtype=np.uint8)
    flags[[2, 7]] = 1
    idx, nf = random_pick(flags, 99, 4)
    assert nf == 2 and sorted(idx[:2]) == [2, 7] and list(idx[2:]) == [-1, -1]
    np.testing.assert_array_equal(random_pick(flags, 99, 4)[0], idx)
    assert random_pick(np.zeros(5), 1, 3)[1] == 0
