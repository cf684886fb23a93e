"""The suggestion step of Algorithm 1, SUGGEST(k, O, RF, Delta), end to end
(the workflow of Sec. 4.1, steps 3-6).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Given every observation so far (configuration, objective values, and whether
the engine ran), in the paper's order:

1. the surrogate sees only the valid observations (Sec. 4.7: crashes are left
   to the forest, so the GP is not distorted by penalty values); each
   objective is standardised over them (mean 0, standard deviation 1; a
   constant objective keeps scale 1), which changes no ranking that follows;
2. each objective's GP hyperparameters are learned by maximum likelihood
   (Sec. 4.3) within the given box, and the GP is fitted (Eq. 4-5);
3. the random forest is trained on every observation with label 1 = ran,
   0 = crashed (Sec. 4.7, Algorithm 1's TRAIN) and read as Q16 votes;
4. the solver's candidates are a Sobol pool on the space's grids, pruned by
   the known constraints (Sec. 4.5.3) and by POF >= Delta (Eq. 3);
5. one objective: MACE -- the Pareto front of UCB, PI and EI and a random
   pick of k from it (Sec. 4.5.1, 4.6); several: the k largest EHVI (Sec.
   4.5.2, 4.6), the reference point standardised like the objectives;
6. a shortfall is made up with Sobol points (Sec. 4.7, last paragraph): the
   pool's points in sequence order that satisfy the known constraints and
   were not picked.  With no valid observation every point comes from here.
"""
import numpy as np

from .forest import feasibility_mask, forest_votes
from .forest_train import train_forest, voting_format
from .gp import gp_fit, gp_posterior
from .hypervolume import ehvi, nondominated
from .mace import mace_suggest, ucb_beta
from .mle import fit_hyperparameters, fit_hyperparameters_warp
from .select import top_q
from .sobol import known_constraints_mask, sobol_pool

DEFAULT_LOWER = (0.01, 0.05, 1e-6)   # lengthscale, signal variance, noise variance
DEFAULT_UPPER = (10.0, 20.0, 1.0)
DEFAULT_START = (0.5, 1.0, 1e-3)


def _box(values, defaults, p, d):
    if values is not None:
        return np.asarray(values, dtype=np.float64).reshape(p, d + 2)
    row = np.log(np.array([defaults[0]] * d + [defaults[1], defaults[2]]))
    return np.tile(row, (p, 1))


WARP_LOWER, WARP_UPPER = 0.2, 5.0   # box of each learned Kumaraswamy parameter


def suggest(X_obs, Y_obs, valid, space, k, delta=0.5, pool_size=4096, pool_skip=0, kernel="matern52",
            warp=None, theta_lower=None, theta_upper=None, theta_start=None, n_trees=16, max_depth=6,
            forest_seed=0, bootstrap=True, xi=1e-4, t=1, pick_seed=0, ref=None, learn_warp=False):
    """Returns dict(x (n_out, d), source (n_out,) 0 = acquisition / 1 = fill,
    theta (p, d + 2), idx (pool indices), and the intermediates).

    learn_warp: the input warping is learned with the other hyperparameters
    (Sec. 4.3, the paper's Matern-3/2 with input warping): each objective's
    search runs over (log l, log s^2, log tau^2, log a, log b) with the warp
    parameters in [WARP_LOWER, WARP_UPPER], starting from ``warp`` (else the
    identity a = b = 1), and theta is then (p, 3d + 2)."""
    levels = np.asarray(space["levels"])
    d = len(levels)
    X_obs = np.asarray(X_obs, dtype=np.float64).reshape(-1, d)
    n_obs = len(X_obs)
    Y_obs = np.asarray(Y_obs, dtype=np.float64)
    p = Y_obs.shape[1] if Y_obs.ndim == 2 else 1
    Y_obs = Y_obs.reshape(n_obs, p)
    ok = np.asarray(valid).reshape(n_obs) != 0

    # 4. candidates and the known constraints
    pool = sobol_pool(space["poly"], space["vinit"], levels, pool_size, pool_skip)
    if space.get("A") is not None and len(np.atleast_1d(space["b"])) > 0:
        known = known_constraints_mask(pool, space["A"], space["b"])
    else:
        known = np.ones(pool_size, dtype=np.uint8)

    out = dict(pool=pool, known=known, theta=np.full((p, 3 * d + 2 if learn_warp else d + 2), np.nan))
    picked = []
    Xv, Yv = X_obs[ok], Y_obs[ok]
    if len(Xv) > 0:
        # 1. standardise the valid observations
        mean = Yv.mean(axis=0)
        sd = Yv.std(axis=0)
        scale = np.where(sd > 0, sd, 1.0)
        Ys = (Yv - mean) / scale
        # 2. hyperparameters and GPs
        lo, hi = _box(theta_lower, DEFAULT_LOWER, p, d), _box(theta_upper, DEFAULT_UPPER, p, d)
        start = np.clip(_box(theta_start, DEFAULT_START, p, d), lo, hi)
        fits = []
        for j in range(p):
            wj = None if warp is None else (np.asarray(warp[0]).reshape(p, d)[j], np.asarray(warp[1]).reshape(p, d)[j])
            th = start[j].copy()
            if learn_warp:
                w0 = (np.ones(d), np.ones(d)) if wj is None else wj
                wlo, whi = np.full(2 * d, np.log(WARP_LOWER)), np.full(2 * d, np.log(WARP_UPPER))
                thw = np.clip(np.concatenate([th, np.log(w0[0]), np.log(w0[1])]),
                              np.concatenate([lo[j], wlo]), np.concatenate([hi[j], whi]))
                thw, _ = fit_hyperparameters_warp(Xv, Ys[:, j], thw, np.concatenate([lo[j], wlo]),
                                                  np.concatenate([hi[j], whi]), kernel)
                out["theta"][j] = thw
                th, wj = thw[:d + 2], (np.exp(thw[d + 2:2 * d + 2]), np.exp(thw[2 * d + 2:]))
            elif np.any(lo[j] != hi[j]):
                th, _ = fit_hyperparameters(Xv, Ys[:, j], th, lo[j], hi[j], kernel, wj)
            if not learn_warp:
                out["theta"][j] = th
            fits.append(gp_fit(Xv, Ys[:, j], np.exp(th[:d]), np.exp(th[d]), np.exp(th[d + 1]), 0.0, kernel=kernel,
                               warp=wj))
        # 3. the forest on every observation
        forest = voting_format(train_forest(X_obs, ok.astype(np.float64), n_trees, max_depth, forest_seed,
                                            bootstrap))
        votes = forest_votes(forest, pool)
        mask = (feasibility_mask(votes, delta, n_trees) & known).astype(np.uint8)
        # 5. score and pick
        P64 = pool.astype(np.float64)
        mu = np.empty((pool_size, p))
        sigma = np.empty((pool_size, p))
        for j, f in enumerate(fits):
            mu[:, j], sigma[:, j] = gp_posterior(f, P64)
        if p == 1:
            res = mace_suggest(mu[:, 0], sigma[:, 0], mask, Ys[:, 0].min(), xi, ucb_beta(t), pick_seed, k)
            idx = res["idx"]
            out.update(res)
        else:
            r = (np.asarray(ref, dtype=np.float64) - mean) / scale if ref is not None else \
                Ys.max(axis=0) + 0.1 * (Ys.max(axis=0) - Ys.min(axis=0))
            front = nondominated(Ys, r)
            acq = ehvi(mu, sigma, front, r)
            idx, val, n_valid = top_q(acq, mask, k)
            out.update(acq=acq, ref=r, front_points=front, val=val, n_valid=n_valid)
        out.update(mu=mu, sigma=sigma, votes=votes, mask=mask)
        picked = [int(i) for i in idx if i >= 0]
    n_solver = len(picked)
    # 6. Sobol fill
    taken = set(picked)
    for i in range(pool_size):
        if len(picked) >= k:
            break
        if known[i] and i not in taken:
            picked.append(i)
    out["idx"] = np.array(picked, dtype=np.int64)
    out["x"] = pool[picked].astype(np.float64) if picked else np.zeros((0, d))
    out["source"] = np.array([0] * n_solver + [1] * (len(picked) - n_solver), dtype=np.int32)
    return out
