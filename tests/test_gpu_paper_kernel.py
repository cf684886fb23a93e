"""GPU parity of the paper's own covariance (Sec. 4.3): Matern-3/2 with
Kumaraswamy input warping, through every call that evaluates the GP
(posterior, the fused scoring pass, the Kriging believer, MACE), against the
oracle.  Tolerances as in test_gpu_parity."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2408_04323_amd as S  # noqa: E402
from oracle.forest import feasibility_mask, forest_votes  # noqa: E402
from oracle.gp import gp_fit, gp_posterior  # noqa: E402
from oracle.pipeline import score_pool as oracle_score_pool  # noqa: E402
from tests.oracle_checks import check_believer, check_mace_front_and_pick  # noqa: E402
from workloads import make_workload  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL = {S.F32: dict(mu=1e-4, sd=1e-3, acq=1e-3), S.F64: dict(mu=1e-10, sd=1e-10, acq=1e-10)}


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def assert_close(got, want, rtol, scale, what):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    bound = rtol * np.maximum(np.abs(want), scale)
    err = np.abs(got - want)
    bad = ~(err <= bound)
    assert not bad.any(), f"{what}: {bad.sum()} of {len(got)} outside tolerance, worst at {np.argmax(err / bound)}"


def dev(a, dtype=torch.float32):
    return torch.as_tensor(np.ascontiguousarray(a)).to(dtype).to(DEV)


_WL = {}


def wl(cfg, n, m=None, warp=True):
    key = (cfg, n, m, warp)
    if key not in _WL:
        _WL[key] = make_workload(cfg, n=n, m=m, kernel="matern32", warp=warp)
    return _WL[key]


def _fits(w, dt):
    warps = w.get("warp")
    out = []
    for j in range(w["p"]):
        wa, wb = (None, None) if warps is None else (warps[0][j], warps[1][j])
        out.append(S.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], w["signal_var"][j], w["noise_var"][j],
                            w["prior_mean"][j], dtype=dt, kernel="matern32", warp_a=wa, warp_b=wb))
    return out


def _oracle_fit(w, j):
    warps = w.get("warp")
    return gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], w["signal_var"][j], w["noise_var"][j],
                  w["prior_mean"][j], kernel="matern32",
                  warp=None if warps is None else (warps[0][j], warps[1][j]))


CASES = [("cfg2-warp", 2, 8192 + 37, None, 0, True), ("cfg3-obj1-warp", 3, 4096 + 5, None, 1, True),
         ("cfg4-obj2-warp", 4, 2048 + 17, None, 2, True), ("cfg2-nowarp", 2, 4096, None, 0, False),
         ("m33-warp", 2, 257, 33, 0, True)]


@pytest.mark.parametrize("dt", [S.F32, S.F64], ids=["f32", "f64"])
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_posterior_matern32_warped(case, dt):
    name, cfg, n, m, obj, warp = case
    w = wl(cfg, n, m, warp)
    say("posterior matern32", name, dt)
    fit = _oracle_fit(w, obj)
    mu_o, sd_o = gp_posterior(fit, w["Xc"].astype(np.float64))
    g = _fits(w, dt)[obj]
    mu, sd = S.posterior(g, dev(w["Xc"]))
    torch.cuda.synchronize()
    t = TOL[dt]
    assert_close(mu.cpu().numpy(), mu_o, t["mu"], np.max(np.abs(mu_o)), f"{name} mu")
    assert_close(sd.cpu().numpy(), sd_o, t["sd"], np.sqrt(w["signal_var"][obj]), f"{name} sigma")
    if warp:  # the warping is live: without it the answer moves
        mu0, _ = gp_posterior(gp_fit(w["X"], w["Y"][:, obj], w["lengthscale"][obj], w["signal_var"][obj],
                                     w["noise_var"][obj], w["prior_mean"][obj], kernel="matern32"),
                              w["Xc"][:64].astype(np.float64))
        assert np.max(np.abs(mu0 - mu_o[:64])) > 100 * t["mu"] * np.max(np.abs(mu_o))


@pytest.mark.parametrize("cfg,n,dt", [(3, 8192, S.F32), (1, 4096, S.F64), (4, 4096, S.F32)])
def test_score_pool_matern32_warped(cfg, n, dt):
    w = wl(cfg, n)
    ref = oracle_score_pool(w)
    gps = _fits(w, dt)
    fd = w["forest"]
    f = S.forest_create(fd["feature"], fd["threshold"], fd["left"], fd["right"], fd["leaf_q16"], fd["tree_offset"],
                        w["d"])
    say("score_pool matern32", cfg, n, dt)
    b = S.score_pool(gps, f, dev(w["Xc"]), w["q"], best_y=w["best_y"], xi=w["xi"], Y_obs=w["Y"],
                     ref=w.get("ref"), delta=w["delta"])
    torch.cuda.synchronize()
    t = TOL[dt]
    for j in range(w["p"]):
        assert_close(b.mu[j].cpu().numpy(), ref["mu"][:, j], t["mu"], np.max(np.abs(ref["mu"][:, j])), f"mu{j}")
        assert_close(b.sigma[j].cpu().numpy(), ref["sigma"][:, j], t["sd"], 1.0, f"sigma{j}")
    assert_close(b.acq.cpu().numpy(), ref["acq"], t["acq"], np.max(ref["acq"]), "acq")
    np.testing.assert_array_equal(b.mask.cpu().numpy(), ref["mask"])
    q = w["q"]
    acq_o = np.where(ref["mask"] != 0, ref["acq"], -np.inf)
    order = np.lexsort((np.arange(len(acq_o)), -acq_o))
    tol = t["acq"] * np.max(ref["acq"])
    for i in b.idx.cpu().numpy():
        assert ref["mask"][i] == 1 and acq_o[i] >= acq_o[order[q - 1]] - 2 * tol


def test_believer_matern32_warped():
    n, m, q = 2048 + 7, 40, 5
    w = wl(5, n, m)
    gps = _fits(w, S.F32)
    fd = w["forest"]
    f = S.forest_create(fd["feature"], fd["threshold"], fd["left"], fd["right"], fd["leaf_q16"], fd["tree_offset"],
                        w["d"])
    say("believer matern32", n, m, q)
    picks, acq_g = S.suggest_kb(gps, f, dev(w["Xc"]), q, w["Y"], w["ref"], delta=w["delta"])
    torch.cuda.synchronize()
    assert len(picks) == q and len(set(picks.tolist())) == q
    mask = feasibility_mask(forest_votes(fd, w["Xc"]), w["delta"], len(fd["tree_offset"]) - 1)
    hyp = [dict(lengthscale=w["lengthscale"][j], signal_var=w["signal_var"][j], noise_var=w["noise_var"][j],
                prior_mean=w["prior_mean"][j], kernel="matern32", warp=(w["warp"][0][j], w["warp"][1][j]))
           for j in range(2)]
    check_believer(w, q, picks, acq_g, mask, hyp=hyp)


def test_mace_matern32_warped():
    from oracle.mace import mace_scores, ucb_beta
    w = wl(1, 4096)
    gp = _fits(w, S.F32)[0]
    fd = w["forest"]
    f = S.forest_create(fd["feature"], fd["threshold"], fd["left"], fd["right"], fd["leaf_q16"], fd["tree_offset"],
                        w["d"])
    beta, seed = ucb_beta(5), 31
    say("mace matern32")
    b = S.suggest_mace(gp, f, dev(w["Xc"]), 4, w["best_y"], beta, seed, xi=w["xi"], delta=w["delta"])
    torch.cuda.synchronize()
    mu_o, sd_o = gp_posterior(_oracle_fit(w, 0), w["Xc"].astype(np.float64))
    assert_close(b.mu.cpu().numpy(), mu_o, 1e-4, np.max(np.abs(mu_o)), "mu")
    u, p, e = (t.cpu().numpy().astype(np.float64) for t in (b.ucb, b.pi, b.ei))
    u_o, p_o, e_o = mace_scores(mu_o, sd_o, w["best_y"], w["xi"], beta)
    assert np.all(np.abs(e - e_o) <= 1e-3 * np.max(e_o))
    mask_o = feasibility_mask(forest_votes(fd, w["Xc"]), w["delta"], len(fd["tree_offset"]) - 1)
    np.testing.assert_array_equal(b.mask.cpu().numpy(), mask_o)
    tol = np.array([1e-3 * max(1.0, beta) * max(1.0, np.max(np.abs(mu_o))), 1e-2, 1e-3 * np.max(e_o)])
    check_mace_front_and_pick(b.front.cpu().numpy(), b.idx.cpu().numpy(), np.stack([u_o, p_o, e_o], 1), mask_o,
                              seed, 4, tol)
