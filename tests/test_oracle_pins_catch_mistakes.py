"""The oracle's pins catch plausible mistakes.  Each case plants one mistake in
a copy of an oracle function (a wrong constant, a dropped term, a flipped
sign, a transposed operand, a strict comparison, the wrong tie order), swaps
it in for the real one, and runs the pin that should notice: the pin must
fail.  Nothing here touches the library; the real oracle is restored after
each case."""
import json
import math
import os

import numpy as np
import pytest
from scipy.linalg import solve_triangular
from scipy.spatial.distance import cdist
from scipy.special import ndtr

import oracle.acquisition as acq
import oracle.forest as forest
import oracle.gp as gp
import oracle.hypervolume as hv
import oracle.mace as mace
import oracle.mle as mle
import oracle.select as select
import test_oracle_acq as pins_acq
import test_oracle_forest_select as pins_forest
import test_oracle_gp as pins_gp
import test_oracle_mace as pins_mace
import test_oracle_mle as pins_mle


@pytest.fixture(scope="module")
def textbook(golden_dir):
    with open(os.path.join(golden_dir, "textbook_values.json")) as fh:
        return json.load(fh)


def _swap(monkeypatch, name, fn, *modules):
    for mod in modules:
        monkeypatch.setattr(mod, name, fn)


def _must_fail(pin, *args):
    with pytest.raises(AssertionError):
        pin(*args)


# ---------------------------------------------------------------- GP (Eq. 4-5)

def test_matern52_wrong_constant(monkeypatch):
    def matern52(A, B, lengthscale, signal_var):  # 5/2 where 5/3 belongs
        r = cdist(np.asarray(A) / lengthscale, np.asarray(B) / lengthscale)
        s5 = math.sqrt(5.0)
        return signal_var * (1.0 + s5 * r + 2.5 * r * r) * np.exp(-s5 * r)
    _swap(monkeypatch, "matern52", matern52, gp, pins_gp)
    _must_fail(pins_gp.test_matern52_matches_sklearn)


def _posterior(fit, Xc, mistake):
    Ks = gp._cross(fit, np.asarray(Xc, dtype=np.float64))
    mu = Ks @ fit["alpha"] + (0.0 if mistake == "no prior mean" else fit["prior_mean"])
    L = fit["L"]
    V = solve_triangular(L.T, Ks.T, lower=False) if mistake == "transposed factor" else \
        solve_triangular(L, Ks.T, lower=True)
    var = fit["signal_var"] - np.sum(V * V, axis=0)
    if mistake == "noisy variance":
        var = var + fit["noise_var"]
    return mu, np.sqrt(np.maximum(var, 0.0))


@pytest.mark.parametrize("mistake,pin", [
    ("no prior mean", "test_single_observation_closed_form"),
    ("noisy variance", "test_posterior_matches_sklearn"),
    ("transposed factor", "test_posterior_matches_sklearn"),
])
def test_posterior_mistakes(monkeypatch, mistake, pin):
    _swap(monkeypatch, "gp_posterior", lambda fit, Xc, chunk=8192: _posterior(fit, Xc, mistake), gp, pins_gp)
    _must_fail(getattr(pins_gp, pin))


# ------------------------------------------------------------ EI (Eq. 8)

def test_partial_expectation_flipped_sign(monkeypatch, textbook):
    def partial_expectation(c, mu, sigma):  # - sigma phi(u) where + belongs
        c, mu, sigma = np.broadcast_arrays(*(np.asarray(v, dtype=np.float64) for v in (c, mu, sigma)))
        u = (c - mu) / sigma
        return (c - mu) * ndtr(u) - sigma * acq.norm_pdf(u)
    _swap(monkeypatch, "partial_expectation", partial_expectation, acq, pins_acq)
    _must_fail(pins_acq.test_partial_expectation_table, textbook)


def test_ei_xi_sign(monkeypatch):
    def expected_improvement(mu, sigma, best_y, xi=acq.XI_PAPER):  # best - xi where best + xi belongs
        return acq.partial_expectation(best_y - xi, mu, sigma)
    _swap(monkeypatch, "expected_improvement", expected_improvement, acq, pins_acq)
    _must_fail(pins_acq.test_ei_monte_carlo_with_xi)


# ----------------------------------------------------------- EHVI (Eq. 9)

def _ehvi(mu, sigma, P, ref, mistake, boxes="columns", chunk=4096):
    mu = np.atleast_2d(np.asarray(mu, dtype=np.float64))
    sigma = np.atleast_2d(np.asarray(sigma, dtype=np.float64))
    lo, hi = (hv.column_boxes if boxes == "columns" else hv.nondominated_cells)(P, ref)
    if mistake == "last box dropped":
        lo, hi = lo[:-1], hi[:-1]
    if mistake == "objectives swapped":
        mu, sigma = mu[:, ::-1], sigma[:, ::-1]
    out = np.zeros(mu.shape[0])
    for b in range(len(lo)):
        term = np.ones(mu.shape[0])
        for j in range(mu.shape[1]):
            term *= acq.partial_expectation(hi[b, j], mu[:, j], sigma[:, j]) - \
                acq.partial_expectation(lo[b, j], mu[:, j], sigma[:, j])
        out += term
    return out


@pytest.mark.parametrize("mistake", ["last box dropped", "objectives swapped"])
def test_ehvi_mistakes(monkeypatch, mistake):
    _swap(monkeypatch, "ehvi", lambda mu, sigma, P, ref, boxes="columns", chunk=4096:
          _ehvi(mu, sigma, P, ref, mistake, boxes), hv, pins_acq)
    _must_fail(pins_acq.test_ehvi_monte_carlo)


# ------------------------------------------------------ forest (Eq. 3)

def test_forest_strict_comparison(monkeypatch):
    def forest_apply(f, Xc):  # x < t where x <= t belongs
        Xc = np.asarray(Xc, dtype=np.float32)
        feat, thr = f["feature"], f["threshold"].astype(np.float32)
        left, right, off = f["left"], f["right"], f["tree_offset"]
        leaves = np.empty((len(Xc), len(off) - 1), dtype=np.int32)
        rows = np.arange(len(Xc))
        for t in range(len(off) - 1):
            node = np.zeros(len(Xc), dtype=np.int64)
            while True:
                internal = left[off[t] + node] >= 0
                if not internal.any():
                    break
                g = off[t] + node[internal]
                node[internal] = np.where(Xc[rows[internal], feat[g]] < thr[g], left[g], right[g])
            leaves[:, t] = node
        return leaves
    _swap(monkeypatch, "forest_apply", forest_apply, forest, pins_forest)
    _must_fail(pins_forest.test_matches_sklearn_forest)


def test_vote_threshold_rounded_down(monkeypatch):
    def vote_threshold(delta, n_trees):  # floor where ceil belongs
        return int(math.floor(float(delta) * float(n_trees * 65536)))
    _swap(monkeypatch, "vote_threshold", vote_threshold, forest, pins_forest)
    _must_fail(pins_forest.test_vote_threshold)


# ------------------------------------------------------- top-q (Sec. 4.6)

def test_top_q_ties_to_highest_index(monkeypatch):
    def top_q(score, mask, q):  # highest index first on ties
        score = np.asarray(score, dtype=np.float64)
        ok = (np.asarray(mask) != 0) & ~np.isnan(score)
        cand = np.arange(len(score))[ok]
        pick = cand[np.lexsort((-cand, -score[cand]))[:q]]
        idx = np.full(q, -1, dtype=np.int64)
        val = np.full(q, np.nan)
        idx[:len(pick)] = pick
        val[:len(pick)] = score[pick]
        return idx, val, int(ok.sum())
    _swap(monkeypatch, "top_q", top_q, select, pins_forest)
    _must_fail(pins_forest.test_top_q_brute_force_and_ties)


# ------------------------------------- hyperparameters (Sec. 4.3) and MACE

def test_nll_log_determinant_doubled(monkeypatch):
    real = mle.nll_and_grad

    def nll_and_grad(theta, X, y, kernel="matern52", warp=None, prior_mean=0.0):  # log det K, not half of it
        nll, grad = real(theta, X, y, kernel, warp, prior_mean)
        d = np.asarray(X).shape[1]
        K = gp.COVARIANCES[kernel](np.asarray(X, dtype=np.float64), np.asarray(X, dtype=np.float64),
                                   np.exp(theta[:d]), np.exp(theta[d])) + np.exp(theta[d + 1]) * np.eye(len(X))
        return nll + 0.5 * np.linalg.slogdet(K)[1], grad
    _swap(monkeypatch, "nll_and_grad", nll_and_grad, mle, pins_mle)
    _must_fail(pins_mle.test_nll_and_gradient_match_sklearn, "matern52", 2.5)


def test_ucb_mean_sign(monkeypatch):
    def ucb_score(mu, sigma, beta):  # + mu where the minimised objective needs - mu
        return beta * np.asarray(sigma, dtype=np.float64) + np.asarray(mu, dtype=np.float64)
    _swap(monkeypatch, "ucb_score", ucb_score, mace, pins_mace)
    _must_fail(pins_mace.test_ucb_score_is_the_mirrored_eq6)


def test_pi_xi_sign(monkeypatch):
    real = mace.probability_of_improvement

    def probability_of_improvement(mu, sigma, best_y, xi):  # best - xi where best + xi belongs
        return real(mu, sigma, best_y - 2 * xi, xi)
    _swap(monkeypatch, "probability_of_improvement", probability_of_improvement, mace, pins_mace)
    _must_fail(pins_mace.test_pi_monte_carlo_with_xi)


def test_front_weak_dominance(monkeypatch):
    def pareto_front_max(scores, mask=None):  # an equal score vector counted as dominating
        S = np.asarray(scores, dtype=np.float64)
        ok = ~np.isnan(S).any(axis=1)
        if mask is not None:
            ok &= np.asarray(mask) != 0
        front = np.zeros(len(S), dtype=bool)
        for i in np.flatnonzero(ok):
            others = np.flatnonzero(ok)
            others = others[others != i]
            front[i] = not (S[others] >= S[i]).all(axis=1).any()
        return front
    _swap(monkeypatch, "pareto_front_max", pareto_front_max, mace, pins_mace)
    _must_fail(pins_mace.test_front_hand_example)


def test_splitmix_wrong_shift(monkeypatch):
    def splitmix64_mix(z):  # 31 where the first shift is 30
        z = (z ^ (z >> 31)) * mace.MIX_M1 & mace.MASK64
        z = (z ^ (z >> 27)) * mace.MIX_M2 & mace.MASK64
        return z ^ (z >> 31)
    monkeypatch.setattr(mace, "splitmix64_mix", splitmix64_mix)
    _must_fail(pins_mace.test_splitmix_reference_outputs)


# ------------------------------------------------ Kriging believer (row A7)

def _believer(X, Y, hypers, Xc, mask, ref, q, mistake, follow=None, record=None):
    X = np.asarray(X, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    Xc64 = np.asarray(Xc, dtype=np.float64)
    p = Y.shape[1]
    Xa, Ya = X.copy(), Y.copy()
    eligible = (np.asarray(mask) != 0).copy()
    picks, vals = [], []
    for _ in range(q):
        mu = np.empty((len(Xc64), p))
        sd = np.empty((len(Xc64), p))
        for j, h in enumerate(hypers):
            fit = gp.gp_fit(Xa, Ya[:, j], h["lengthscale"], h["signal_var"], h["noise_var"], h["prior_mean"])
            mu[:, j], sd[:, j] = gp.gp_posterior(fit, Xc64)
        front = hv.nondominated(Y if mistake == "front not updated" else Ya, ref)
        acq_v = hv.ehvi(mu, sd, front, ref)
        idx, val, _ = select.top_q(acq_v, eligible, 1)
        if idx[0] < 0:
            break
        i = int(idx[0])
        picks.append(i)
        vals.append(float(val[0]))
        if mistake != "pick not excluded":
            eligible[i] = False
        fantasy = Y.min(axis=0) if mistake == "best observed as fantasy" else mu[i]
        Xa = np.vstack([Xa, Xc64[i][None, :]])
        Ya = np.vstack([Ya, fantasy[None, :]])
    return np.array(picks, dtype=np.int64), np.array(vals), mu, sd


# (Leaving the pick eligible is no mistake a pin can see: with its fantasy
# joined, the picked candidate's variance collapses and its mean sits on the
# front, so its EHVI is about zero and it is not picked again.)
@pytest.mark.parametrize("mistake", ["best observed as fantasy", "front not updated"])
def test_believer_mistakes(monkeypatch, mistake):
    import test_oracle_believer as pins_believer
    _swap(monkeypatch, "kriging_believer",
          lambda X, Y, hypers, Xc, mask, ref, q, follow=None, record=None:
          _believer(X, Y, hypers, Xc, mask, ref, q, mistake), pins_believer)
    _must_fail(pins_believer.test_believer_second_step_by_the_downdate)


# ----------------- candidate pool, Delta adaptation, forest training (N3b, N4, A8)

def test_sobol_without_gray_code(monkeypatch):
    import oracle.sobol as sobol
    import test_oracle_sobol as pins_sobol

    def sobol_points(poly, vinit, n, skip=0):  # index i where the Gray code i ^ (i >> 1) belongs
        V = [sobol.direction_numbers(poly[j], vinit[j]) for j in range(len(poly))]
        out = np.zeros((n, len(poly)))
        for r in range(n):
            g = skip + r
            for j in range(len(poly)):
                x, k = 0, 0
                while g >> k:
                    if (g >> k) & 1:
                        x ^= V[j][k]
                    k += 1
                out[r, j] = x / 2.0 ** 32
        return out
    _swap(monkeypatch, "sobol_points", sobol_points, sobol, pins_sobol)
    _must_fail(pins_sobol.test_points_match_scipy, 5, 1024)


def test_delta_steps_the_wrong_way(monkeypatch, golden_dir):
    import oracle.threshold as threshold

    def delta_update(delta, c, k, any_invalid, upsilon=threshold.UPSILON):  # raised where it is lowered
        if any_invalid:
            return min(0.75, max(0.5, delta + upsilon)), 0
        c = c + k
        if c >= 5:
            delta = min(0.75, delta + upsilon)
            c = c - 5
        return delta, c
    _swap(monkeypatch, "delta_update", delta_update, threshold, pins_forest)
    _must_fail(pins_forest.test_delta_sequences, golden_dir)


def test_split_at_the_lower_value(monkeypatch):
    import oracle.forest_train as ft
    import test_oracle_forest_train as pins_ft
    real = ft._grow

    def _grow(X, y, w, idx, depth, max_depth, nodes):  # threshold at the left value, not the midpoint
        me = real(X, y, w, idx, depth, max_depth, nodes)
        f = nodes[me]["feature"]
        if f >= 0:
            xs = np.sort(X[idx, f])
            t = nodes[me]["threshold"]
            nodes[me]["threshold"] = xs[xs <= t].max()
        return me
    monkeypatch.setattr(ft, "_grow", _grow)
    _must_fail(pins_ft.test_single_tree_matches_sklearn, 1, 6)


# --------------------------------------- the voting format (Eq. 3, Sec. 4.7)

def _voting_format(tf, mistake):
    t64 = np.asarray(tf["threshold"], dtype=np.float64)
    t32 = t64.astype(np.float32)
    if mistake != "threshold to nearest":
        above = t32.astype(np.float64) > t64
        t32[above] = np.nextafter(t32[above], np.float32(-np.inf))
    leaf = np.asarray(tf["left"]) < 0
    v = np.asarray(tf["value"]) * 65536.0
    q = {"leaf half up": np.floor(v + 0.5), "leaf truncated": np.floor(v)}.get(mistake, np.rint(v))
    return dict(feature=np.where(leaf, 0, tf["feature"]).astype(np.int32),
                threshold=np.where(leaf, np.float32(0), t32).astype(np.float32),
                left=np.asarray(tf["left"], np.int32), right=np.asarray(tf["right"], np.int32),
                leaf_q16=np.where(leaf, q, 0).astype(np.int32), tree_offset=np.asarray(tf["tree_offset"], np.int64))


@pytest.mark.parametrize("mistake,pin,args", [
    ("threshold to nearest", "test_voting_format_threshold_is_the_float32_below", (0.3 - 1e-9, None)),
    ("threshold to nearest", "test_voting_format_votes_match_the_float64_walk", ()),
    ("leaf half up", "test_voting_format_leaf_q16_ties_to_even", (2.5 / 65536, 2)),
    ("leaf truncated", "test_voting_format_leaf_q16_ties_to_even", (1.5 / 65536, 2)),
])
def test_voting_format_mistakes(monkeypatch, mistake, pin, args):
    import test_oracle_forest_train as pins_ft
    if args and args[1] is None:    # a float64 threshold just below float32(0.3): the float32 below it
        args = (float(np.float32(0.3)) - 1e-12, float(np.nextafter(np.float32(0.3), np.float32(0))))
    monkeypatch.setattr(pins_ft, "voting_format", lambda tf: _voting_format(tf, mistake))
    _must_fail(getattr(pins_ft, pin), *args)


# ---------------------------------- the whole scoring pass (Sec. 4.1, 3-8)

def _score_pool(w, mistake):
    from oracle.acquisition import expected_improvement
    from oracle.forest import feasibility_mask, forest_votes
    from oracle.hypervolume import ehvi, nondominated
    p = w["Y"].shape[1]
    fits = []
    for j in range(p):
        h = 0 if mistake == "first objective's hyperparameters" else j
        fits.append(gp.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][h], w["signal_var"][h], w["noise_var"][h],
                              w["prior_mean"][h]))
    Xc = w["Xc"]
    mu = np.empty((len(Xc), p))
    sigma = np.empty((len(Xc), p))
    for j, f in enumerate(fits):
        mu[:, j], sigma[:, j] = gp.gp_posterior(f, Xc)
    front = None
    if p == 1:
        acq_ = expected_improvement(mu[:, 0], sigma[:, 0], w["best_y"], w["xi"])
    else:
        front = nondominated(w["Y"], w["ref"])
        acq_ = ehvi(mu, sigma, front, w["ref"])
    votes = forest_votes(w["forest"], Xc)
    T = len(w["forest"]["tree_offset"]) - (0 if mistake == "tree count off by one" else 1)
    mask = feasibility_mask(votes, w["delta"], T)
    if mistake == "mask ignored":
        mask = np.ones_like(mask)
    idx, val, n_valid = select.top_q(acq_, mask, w["q"])
    return dict(mu=mu, sigma=sigma, acq=acq_, front=front, votes=votes, mask=mask, idx=idx, val=val,
                n_valid=n_valid)


@pytest.mark.parametrize("mistake,pin,args", [
    ("first objective's hyperparameters", "test_two_objective_pass_by_hand", ([1.0, 1.0], 1)),
    ("mask ignored", "test_single_objective_pass_by_hand", ()),
    ("tree count off by one", "test_single_objective_pass_by_hand", ()),
])
def test_score_pool_mistakes(monkeypatch, mistake, pin, args):
    import test_oracle_pipeline as pins_pipe
    monkeypatch.setattr(pins_pipe, "score_pool", lambda w, Xc=None: _score_pool(w, mistake))
    _must_fail(getattr(pins_pipe, pin), *args)


# -------------------------------- learned input warping (Sec. 4.3, Snoek et al.)

def _warp_derivatives(X, a, b, mistake):
    X = np.clip(np.asarray(X, dtype=np.float64), 0.0, 1.0)
    inner = (X > 0) & (X < 1)
    Xi = np.where(inner, X, 0.5)
    u = Xi ** a
    w = 1.0 - (1.0 - X ** a) ** b
    fa = 1.0 if mistake == "derivative in a, not log a" else a
    da = np.where(inner, fa * b * (1.0 - u) ** (b - 1.0) * u * np.log(Xi), 0.0)
    sb = 1.0 if mistake == "sign of the b derivative" else -1.0
    db = np.where(inner, sb * b * (1.0 - u) ** b * np.log(1.0 - u), 0.0)
    return w, da, db


@pytest.mark.parametrize("mistake", ["derivative in a, not log a", "sign of the b derivative"])
def test_warp_gradient_mistakes(monkeypatch, mistake):
    monkeypatch.setattr(mle, "warp_derivatives", lambda X, a, b: _warp_derivatives(X, a, b, mistake))
    _must_fail(pins_mle.test_warp_gradient_matches_finite_differences, "matern32")
