"""One whole scoring pass of the suggestion step over a candidate pool
(workflow steps 3-8 of Sec. 4.1): GP posterior per objective (Eq. 4-5), the
acquisition (EI, Eq. 8, for one objective; EHVI, Eq. 9, for several), the
random-forest mask POF >= Delta (Eq. 3) and the top-q pick (Sec. 4.6)."""
import numpy as np

from .acquisition import expected_improvement
from .forest import feasibility_mask, forest_votes
from .gp import gp_fit, gp_posterior
from .hypervolume import ehvi, nondominated
from .select import top_q


def score_pool(w, Xc=None):
    """``w`` is a workload dict from the seeded generators.  Returns a dict of
    every intermediate (fits, mu, sigma, acq, votes, mask, idx, val, n_valid)."""
    Xc = w["Xc"] if Xc is None else Xc
    p = w["Y"].shape[1]
    warps = w.get("warp")
    fits = [gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], w["signal_var"][j],
                   w["noise_var"][j], w["prior_mean"][j], kernel=w.get("kernel", "matern52"),
                   warp=None if warps is None else (warps[0][j], warps[1][j])) for j in range(p)]
    mu = np.empty((len(Xc), p))
    sigma = np.empty((len(Xc), p))
    for j, f in enumerate(fits):
        mu[:, j], sigma[:, j] = gp_posterior(f, Xc)
    if p == 1:
        acq = expected_improvement(mu[:, 0], sigma[:, 0], w["best_y"], w["xi"])
        front = None
    else:
        front = nondominated(w["Y"], w["ref"])
        acq = ehvi(mu, sigma, front, w["ref"])
    votes = forest_votes(w["forest"], Xc)
    mask = feasibility_mask(votes, w["delta"], len(w["forest"]["tree_offset"]) - 1)
    idx, val, n_valid = top_q(acq, mask, w["q"])
    return dict(fits=fits, mu=mu, sigma=sigma, acq=acq, front=front, votes=votes,
                mask=mask, idx=idx, val=val, n_valid=n_valid)
