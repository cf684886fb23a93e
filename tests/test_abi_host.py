"""CPU tests of the C ABI: every declared symbol is exported, and the host-side
logic (fit arithmetic, front, Delta update, vote threshold, argument checks)
agrees with the oracle.  No device compute runs here."""
import ctypes as C
import json
import os
import re

import numpy as np
import pytest

import paper_2408_04323_amd as S
from paper_2408_04323_amd._native import SIGNATURES, lib
from oracle.forest import vote_threshold as oracle_vote_threshold
from oracle.gp import gp_fit as oracle_fit
from oracle.hypervolume import nondominated
from oracle.threshold import delta_update as oracle_delta

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    with open(os.path.join(ROOT, "include", "scoot.h")) as fh:
        text = fh.read()
    return sorted(set(re.findall(r"^(?:int|const char\*)\s+(scoot_\w+)\(", text, re.M)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert len(names) >= 17
    L = lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(SIGNATURES)
    assert S.abi_version() == 5


def test_factor_matches_oracle():
    rng = np.random.default_rng(1)
    X = rng.random((40, 7))
    y = rng.standard_normal(40)
    ls = rng.uniform(0.2, 1.0, 7)
    L, alpha = S.gp_factor_host(X, y, ls, 1.3, 1e-3, 0.25)
    f = oracle_fit(X, y, ls, 1.3, 1e-3, 0.25)
    np.testing.assert_allclose(L, f["L"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(alpha, f["alpha"], rtol=1e-10, atol=1e-10)


def test_factor_matern32_warped_matches_oracle():
    rng = np.random.default_rng(2)
    X = rng.random((40, 7))
    y = rng.standard_normal(40)
    ls = rng.uniform(0.2, 1.0, 7)
    a = np.exp(0.5 * rng.standard_normal(7))
    b = np.exp(0.5 * rng.standard_normal(7))
    L, alpha = S.gp_factor_host(X, y, ls, 0.8, 1e-3, -0.1, kernel="matern32", warp_a=a, warp_b=b)
    f = oracle_fit(X, y, ls, 0.8, 1e-3, -0.1, kernel="matern32", warp=(a, b))
    np.testing.assert_allclose(L, f["L"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(alpha, f["alpha"], rtol=1e-10, atol=1e-10)
    # Matern-3/2 without warping, too
    L2, _ = S.gp_factor_host(X, y, ls, 0.8, 1e-3, kernel="matern32")
    np.testing.assert_allclose(L2, oracle_fit(X, y, ls, 0.8, 1e-3, kernel="matern32")["L"], rtol=0, atol=1e-12)
    with pytest.raises(S.ScootError):
        S.gp_factor_host(X, y, ls, 0.8, 1e-3, kernel="matern32", warp_a=a, warp_b=-b)
    with pytest.raises(ValueError):
        S.gp_factor_host(X, y, ls, 0.8, 1e-3, warp_a=a)


def test_fit_errors():
    X = np.zeros((3, 2))
    with pytest.raises(S.ScootError) as e:
        S.gp_factor_host(X, np.zeros(3), [1.0, 1.0], 1.0, 0.0)
    assert e.value.status == -2
    with pytest.raises(S.ScootError) as e:
        S.gp_factor_host(np.random.rand(4, 2), np.zeros(4), [1.0, -1.0], 1.0, 1e-3)
    assert e.value.status == -1
    with pytest.raises(S.ScootError) as e:
        S.gp_factor_host(np.random.rand(4, 17), np.zeros(4), np.ones(17), 1.0, 1e-3)
    assert e.value.status == -4
    with pytest.raises(S.ScootError) as e:
        S.gp_factor_host(np.random.rand(577, 2), np.zeros(577), np.ones(2), 1.0, 1e-3)
    assert e.value.status == -4
    y = np.zeros(4)
    y[1] = np.nan
    with pytest.raises(S.ScootError) as e:
        S.gp_factor_host(np.random.rand(4, 2), y, np.ones(2), 1.0, 1e-3)
    assert e.value.status == -1


@pytest.mark.parametrize("p", [1, 2, 3])
def test_front_matches_oracle(p):
    rng = np.random.default_rng(10 + p)
    Y = rng.standard_normal((60, p))
    if p > 1:
        Y[:, 1] = -0.8 * Y[:, 0] + 0.3 * Y[:, 1]
    Y = np.vstack([Y, Y[:5]])  # duplicates
    ref = Y.max(axis=0) + 0.1
    front, n_boxes = S.ehvi_front(Y, ref)
    want = nondominated(Y, ref)
    np.testing.assert_array_equal(front, want)
    if p == 1:
        assert n_boxes == 1
    if p == 2:
        assert n_boxes == len(want) + 1
    if p == 3:
        assert len(want) + 1 <= n_boxes <= (len(want) + 1) ** 2


def test_front_excludes_points_not_below_ref():
    front, nb = S.ehvi_front(np.array([[1.0, 5.0], [2.0, 2.0], [5.0, 1.0]]), np.array([4.0, 4.0]))
    assert front.tolist() == [[2.0, 2.0]] and nb == 2
    front, nb = S.ehvi_front(np.zeros((0, 2)), np.array([1.0, 1.0]))
    assert len(front) == 0 and nb == 1


def test_delta_update_matches_golden(golden_dir):
    with open(os.path.join(golden_dir, "delta_sequences.json")) as fh:
        g = json.load(fh)
    for seq in g["sequences"]:
        d, c = 0.5, 0
        od, oc = 0.5, 0
        for k, bad, want_d, want_c in seq["steps"]:
            d, c = S.delta_update(d, c, k, bad)
            od, oc = oracle_delta(od, oc, k, bad)
            assert d == pytest.approx(want_d, abs=1e-12) and c == want_c
            assert d == od and c == oc


def test_vote_threshold_matches_oracle():
    for delta in [0.0, 0.25, 0.3, 0.45, 0.5, 0.55, 0.6, 0.75, 1.0]:
        for T in [1, 3, 16, 64, 128, 1000]:
            assert S.vote_threshold(delta, T) == oracle_vote_threshold(delta, T)
    with pytest.raises(S.ScootError):
        S.vote_threshold(1.5, 4)


def test_topq_and_forest_argument_checks():
    L = lib()
    idx = C.c_void_p(0)
    assert L.scoot_suggest_topq(None, None, 10, 0, 0, idx, None, None, None) == -1   # q = 0
    assert L.scoot_suggest_topq(None, None, 10, 0, 65, idx, None, None, None) == -1  # q > max
    assert L.scoot_suggest_topq(None, None, -1, 0, 4, idx, None, None, None) == -1
    # a tree whose child points back at the root is not a tree
    with pytest.raises(S.ScootError) as e:
        S.forest_create([0, 0, 0], [0.5, 0, 0], [1, -1, 0], [2, -1, -1], [0, 1, 1], [0, 3], 2)
    assert e.value.status == -1
    with pytest.raises(S.ScootError) as e:  # feature out of range
        S.forest_create([5, 0, 0], [0.5, 0, 0], [1, -1, -1], [2, -1, -1], [0, 1, 1], [0, 3], 2)
    assert e.value.status == -1
    with pytest.raises(S.ScootError) as e:  # leaf value above 1.0 in Q16
        S.forest_create([0, 0, 0], [0.5, 0, 0], [1, -1, -1], [2, -1, -1], [0, 70000, 1], [0, 3], 2)
    assert e.value.status == -1


def test_normal_tail_coefficients_match_their_generator():
    """The float partial expectation uses P4(s) / Q6(s) for g(x) = 1 - x M(x);
    the coefficients in the kernel source must be what the committed fitting
    script produces, and the fit must meet its stated error."""
    import importlib.util
    here = os.path.join(os.path.dirname(S.__file__), "csrc")
    spec = importlib.util.spec_from_file_location("gen_normal_tail", os.path.join(here, "gen_normal_tail.py"))
    gen = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(gen)
    x, y, p, q, err = gen.fit()
    assert err < 2e-8
    src = open(os.path.join(here, "normal.h")).read()
    body = src[src.index("__device__ inline float h_normal(float u)"):]
    body = body[:body.index("\n}\n")]
    nums = [float(v) for v in re.findall(r"([0-9]\.[0-9]{9}e[+-][0-9]{2})f", body)]
    # Horner order: highest coefficient first, P then Q (constant 1 of Q written as 1.0f)
    want = list(p[::-1]) + list(q[:0:-1])
    assert len(nums) == len(want)
    np.testing.assert_allclose(nums, want, rtol=5e-9)
    # the float evaluation of the fit against g in double
    g32 = gen.eval_f32(p, q, x).astype(np.float64)
    assert np.max(np.abs(g32 - y) / y) < 1e-6


def test_sobol_and_known_constraint_argument_checks():
    """Validation happens on the host before any launch (n = 0 launches nothing)."""
    L = lib()
    U32 = C.c_uint32 * 2
    vin = (C.c_uint32 * 36)()
    vin[18] = 1                                       # dim 1: x + 1, m_1 = 1
    lv = (C.c_int32 * 2)(0, 5)

    def call(poly=(1, 3), levels=lv, d=2, skip=0, n=0, A=None, b=None, r=0, v=vin):
        return L.scoot_sobol_pool(U32(*poly), v, d, levels, skip, n, A, b, r, None, None, None)

    assert call() == 0
    assert call(poly=(1, 2)) == -1                   # no constant term
    assert call(poly=(1, 0)) == -1
    assert call(poly=(1, 1 << 20 | 1)) == -4          # degree 20 > 18
    bad = (C.c_uint32 * 36)()
    bad[18] = 2                                       # m_1 must be odd
    assert call(v=bad) == -1
    bad[18] = 3                                       # and below 2^1
    assert call(v=bad) == -1
    assert call(levels=(C.c_int32 * 2)(0, -1)) == -1
    assert call(d=0) == -1 and call(d=17) == -1
    assert call(skip=-1) == -1 and call(n=-1) == -1
    assert call(skip=1 << 32, n=0) == 0 and call(skip=(1 << 32) + 1, n=0) == -1   # skip + n <= 2^32
    assert call(n=10) == -1                           # null Xc
    A = (C.c_double * 18)(*([1.0] * 18))
    b = (C.c_double * 9)(*([1.0] * 9))
    assert call(A=A, b=b, r=9) == -4                  # r > SCOOT_MAX_CONSTRAINTS
    assert call(A=None, b=b, r=1) == -1
    assert call(A=A, b=b, r=-1) == -4
    A[1] = float("inf")
    assert call(A=A, b=b, r=1) == -1
    A[1] = 1.0
    b[0] = float("nan")
    assert call(A=A, b=b, r=1) == -1
    b[0] = float("inf")                               # an always-true row is fine
    assert call(A=A, b=b, r=1) == 0
    K = L.scoot_known_constraints
    assert K(None, 0, 2, A, b, 1, None, None) == 0
    assert K(None, 5, 2, A, b, 1, None, None) == -1
    assert K(None, 0, 0, A, b, 1, None, None) == -1
    assert K(None, 0, 2, A, b, 9, None, None) == -4
    with pytest.raises(ValueError):
        S.sobol_pool([1, 3], [[0], [1]], [0], 4)      # one level per dimension


def test_suggest_argument_checks():
    """scoot_suggest rejects bad arguments before any device work."""
    from tests.suggest_cases import observations, space
    sp = space()
    X, Y, v = observations(6, p=2)
    bad = [dict(k=0), dict(k=65), dict(k=2, delta=1.5), dict(k=2, delta=-0.1), dict(k=2, pool_size=0),
           dict(k=2, pool_size=2 ** 31), dict(k=2, pool_skip=-1), dict(k=2, kernel=7), dict(k=2, dtype=5),
           dict(k=2, n_trees=0), dict(k=2, max_depth=-1), dict(k=2, xi=float("nan")),
           dict(k=2, ref=[0.0, float("inf")]),
           dict(k=2, theta_lower=np.zeros((2, 6)), theta_upper=-np.ones((2, 6)))]
    for kw in bad:
        with pytest.raises(S.ScootError) as e:
            S.suggest(X, Y, v, sp, stream=0, **kw)
        assert e.value.status == -1, kw
    with pytest.raises(ValueError):  # warps go in pairs
        S.suggest(X, Y, v, sp, k=2, warp_a=np.ones((2, 4)), stream=0)
    with pytest.raises(S.ScootError):  # t < 1 with one objective
        S.suggest(X, Y[:, :1], v, sp, k=2, t=0, stream=0)
    with pytest.raises(S.ScootError):  # non-finite observation
        Xn = X.copy()
        Xn[0, 0] = np.nan
        S.suggest(Xn, Y, v, sp, k=2, stream=0)
