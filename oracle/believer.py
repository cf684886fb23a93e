"""Sequential Kriging-believer selection of q candidates (an extension of the
parallel suggestion of Sec. 4.6; the paper itself takes the top k by EHVI).

Written as the plain definition: before every pick the GP of each objective is
refitted from scratch on the observations plus the earlier picks, each pick
carrying the fantasy value y = mu(x_pick) of its own objective's current GP and
the same noise tau^2 as a real observation.  The front is the non-dominated set
of the observed values plus those fantasies; the reference point stays fixed.
Every pick maximises EHVI over the feasible candidates not yet picked (score
descending, lowest index first on ties).
"""
import numpy as np

from .gp import gp_fit, gp_posterior
from .hypervolume import ehvi, nondominated
from .select import top_q


def kriging_believer(X, Y, hypers, Xc, mask, ref, q, follow=None, record=None):
    """hypers: list over objectives of dicts with lengthscale, signal_var,
    noise_var, prior_mean (and optionally kernel, warp as in ``gp_fit``).  Returns (picks (q,), per-pick EHVI (q,),
    final mu (n, p), final sigma (n, p)).

    ``follow``: a pick sequence to take instead of the arg max at each step
    (to check another implementation's greedy sequence step by step);
    ``record``: a list that receives (acq, eligible) of every step."""
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
            fit = gp_fit(Xa, Ya[:, j], h["lengthscale"], h["signal_var"], h["noise_var"], h["prior_mean"],
                         kernel=h.get("kernel", "matern52"), warp=h.get("warp"))
            mu[:, j], sd[:, j] = gp_posterior(fit, Xc64)
        front = nondominated(Ya, ref)
        acq = ehvi(mu, sd, front, ref)
        if record is not None:
            record.append((acq.copy(), eligible.copy()))
        if follow is not None:
            if len(picks) >= len(follow):
                break
            i = int(follow[len(picks)])
            val = [acq[i]]
        else:
            idx, val, _ = top_q(acq, eligible, 1)
            if idx[0] < 0:
                break
            i = int(idx[0])
        picks.append(i)
        vals.append(float(val[0]))
        eligible[i] = False
        Xa = np.vstack([Xa, Xc64[i][None, :]])
        Ya = np.vstack([Ya, mu[i][None, :]])
    return np.array(picks, dtype=np.int64), np.array(vals), mu, sd
