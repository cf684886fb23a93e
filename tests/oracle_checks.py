"""Checks of the library's sequential and randomised suggestions against the
oracle's own runs from the same seeded inputs (the oracle never sees a
library output)."""
import sys

import numpy as np

from oracle.believer import kriging_believer
from oracle.mace import pareto_front_max, random_pick
from oracle.select import top_q


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def check_believer(w, q, picks, acq_g, mask, hyp=None, min_steps=1):
    """The oracle runs its own greedy sequence from the same inputs (a full
    refit per pick).  Step by step, while the two sequences agree, the
    library's pick must be the oracle's where the oracle's best is clear of the
    runner-up by more than twice the bar, and within the bar of it otherwise,
    and its reported EHVI must match.  At a near tie the sequences may part;
    their histories differ from there on, so the comparison stops there; at
    least ``min_steps`` steps must be compared.  Returns (steps compared, the
    oracle's mean (n, p) and deviation (n, p) of its last scoring round); the
    last two describe the library's last round when every step was compared
    and the picks agree."""
    if hyp is None:
        hyp = [dict(lengthscale=w["lengthscale"][j], signal_var=w["signal_var"][j], noise_var=w["noise_var"][j],
                    prior_mean=w["prior_mean"][j]) for j in range(w["p"])]
    steps = []
    picks_o, _, mu_o, sd_o = kriging_believer(w["X"], w["Y"], hyp, w["Xc"], mask, w["ref"], q, record=steps)
    assert len(picks_o) == len(picks)
    compared = 0
    for j, (acq_o, elig) in enumerate(steps):
        tol = 1e-3 * np.max(acq_o[elig != 0])
        i, io = int(picks[j]), int(picks_o[j])
        assert elig[i], f"step {j}: pick {i} not eligible"
        assert acq_o[i] >= acq_o[io] - 2 * tol, f"step {j}: pick {i} has EHVI {acq_o[i]} below the best {acq_o[io]}"
        assert abs(acq_g[j] - acq_o[i]) <= tol + 1e-3 * abs(acq_o[i]), f"step {j}: EHVI {acq_g[j]} vs {acq_o[i]}"
        compared += 1
        if i != io:
            second = np.sort(np.where(elig != 0, acq_o, -np.inf))[::-1][1]
            assert acq_o[io] - second <= 2 * tol, f"step {j}: decided pick {io} but got {i}"
            break
    say("believer steps compared", compared, "of", len(picks))
    assert compared >= min_steps, f"only {compared} believer steps compared, {min_steps} required"
    return compared, mu_o, sd_o


def believer_gaps(w, q, mask, hyp=None):
    """The oracle's own greedy run: at each step, the gap between its best and
    its runner-up in units of the bar (1e-3 of the step's largest eligible
    EHVI).  A gap above 2 everywhere means the whole sequence is decided."""
    if hyp is None:
        hyp = [dict(lengthscale=w["lengthscale"][j], signal_var=w["signal_var"][j], noise_var=w["noise_var"][j],
                    prior_mean=w["prior_mean"][j]) for j in range(w["p"])]
    steps = []
    kriging_believer(w["X"], w["Y"], hyp, w["Xc"], mask, w["ref"], q, record=steps)
    out = []
    for acq_o, elig in steps:
        ranked = np.sort(np.where(elig != 0, acq_o, -np.inf))[::-1]
        out.append((ranked[0] - ranked[1]) / (1e-3 * ranked[0]))
    return out


def check_mace_front_and_pick(front_g, idx_g, scores_o, mask_o, seed, q, tol):
    """front_g, idx_g: the library's front (bool) and picks; scores_o: the
    oracle's (UCB, PI, EI) on the same candidates, mask_o the oracle's mask,
    tol the bar of each score: (3,) for every candidate, or (n, 3) per
    candidate.  Where the two fronts disagree on a candidate, some other
    eligible candidate must sit within the two candidates' bars of dominating
    it (a near tie, not a wrong front).  With equal fronts the picks must be
    the oracle's draw from its front exactly; otherwise each pick must be a
    distinct member of the library's front."""
    fo = pareto_front_max(scores_o, mask_o)
    fg = np.asarray(front_g).astype(bool)
    tol = np.broadcast_to(np.asarray(tol, dtype=np.float64), scores_o.shape)
    elig = np.flatnonzero(np.asarray(mask_o) != 0)
    for i in np.flatnonzero(fg != fo):
        others = elig[elig != i]
        dlt = scores_o[others] - scores_o[i]
        tol2 = tol[others] + tol[i]
        near = (dlt >= -tol2).all(axis=1) & (np.abs(dlt) <= tol2).any(axis=1)
        assert near.any(), f"front disagreement at {i} is not a near tie"
    idx_g = np.asarray(idx_g)
    if np.array_equal(fg, fo):
        want, _ = random_pick(fo, seed, q)
        np.testing.assert_array_equal(idx_g, want)
    else:
        got = idx_g[idx_g >= 0]
        assert len(set(got.tolist())) == len(got) and fg[got].all()
        assert len(got) == min(q, int(fg.sum()))


def check_topq(idx_g, n_valid_g, acq_o, mask_o, q, rtol):
    """The library's top-q picks against the oracle's ranking of its own
    scores: the eligible count exact; the picks exactly the oracle's set where
    its cut between ranks q and q + 1 is clear by more than twice the bar
    (rtol times the largest eligible score), and every pick eligible and
    within twice the bar of the oracle's q-th best otherwise."""
    want_idx, want_val, want_nv = top_q(acq_o, mask_o, q)
    assert int(n_valid_g) == want_nv
    idx_g = np.asarray(idx_g)
    if want_nv == 0:
        assert np.all(idx_g == -1)
        return
    elig = np.where(np.asarray(mask_o) != 0, acq_o, -np.inf)
    tol = rtol * np.max(np.abs(elig[np.isfinite(elig)]))
    k = min(q, want_nv)
    kth = want_val[k - 1]
    nxt = np.sort(elig)[::-1][k] if want_nv > k else -np.inf
    got = idx_g[:k]
    assert np.all(idx_g[k:] == -1)
    if kth - nxt > 2 * tol:
        assert set(got.tolist()) == set(want_idx[:k].tolist())
    for i in got:
        assert np.asarray(mask_o)[i] != 0 and acq_o[i] >= kth - 2 * tol
