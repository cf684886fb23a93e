"""GPU parity of every step of the scoring path against the oracle.

Float results: |gpu - oracle| <= rtol * max(|oracle|, scale) element by
element, rtol = 1e-4 (mu) and 1e-3 (sigma, EI, EHVI) in float32, 1e-10 in
float64; scale = max |mu| over the pool for mu, the signal standard deviation
for sigma, the largest oracle value of the pool for EI and EHVI.
Integer results (leaf ids, votes, mask, top-q indices on a shared score array)
are bit-exact.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2408_04323_amd as S  # noqa: E402
from oracle.acquisition import expected_improvement  # noqa: E402
from oracle.forest import feasibility_mask, forest_apply, forest_votes  # noqa: E402
from oracle.gp import gp_fit, gp_posterior  # noqa: E402
from oracle.hypervolume import ehvi as oracle_ehvi, nondominated  # noqa: E402
from oracle.pipeline import score_pool as oracle_score_pool  # noqa: E402
from oracle.select import top_q  # noqa: E402
from tests.oracle_checks import check_believer, check_topq  # noqa: E402
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
    assert got.shape == want.shape, what
    bound = rtol * np.maximum(np.abs(want), scale)
    err = np.abs(got - want)
    bad = ~(err <= bound)
    assert not bad.any(), (f"{what}: {bad.sum()} of {len(got)} outside tolerance; worst "
                           f"{np.max(err / np.maximum(bound, 1e-300)):.3g}x bound at {np.argmax(err / bound)}")


def as_held(a, dtype):
    """A seeded input as the device holds it (rounded on the host)."""
    return np.asarray(a).astype(np.float32 if dtype == torch.float32 else np.float64).astype(np.float64)


def dev(a, dtype=torch.float32):
    return torch.as_tensor(np.ascontiguousarray(a)).to(dtype).to(DEV)


_WL = {}


def wl(cfg, n, m=None):
    key = (cfg, n, m)
    if key not in _WL:
        _WL[key] = make_workload(cfg, n=n, m=m)
    return _WL[key]


# --------------------------------------------------------------------------- posterior
POST_CASES = [
    ("cfg1", 1, 4096, None, 0),
    ("cfg2-ragged", 2, 8192 + 37, None, 0),
    ("cfg3-obj0", 3, 4096 + 5, None, 0),
    ("cfg3-obj1", 3, 4096 + 5, None, 1),
    ("cfg4-obj2", 4, 2048 + 17, None, 2),
    ("cfg5-m520", 5, 2048 + 3, 520, 0),
    ("m33-ragged-obs", 2, 257, 33, 0),
]


@pytest.mark.parametrize("dt", [S.F32, S.F64], ids=["f32", "f64"])
@pytest.mark.parametrize("case", POST_CASES, ids=[c[0] for c in POST_CASES])
def test_posterior_parity(case, dt):
    name, cfg, n, m, obj = case
    w = wl(cfg, n, m)
    say("posterior", name, "dtype", dt, "m", w["m"], "n", n)
    args = (w["X"], w["Y"][:, obj], w["lengthscale"][obj], w["signal_var"][obj], w["noise_var"][obj],
            w["prior_mean"][obj])
    fit = gp_fit(*args)
    mu_o, sd_o = gp_posterior(fit, w["Xc"].astype(np.float64))
    g = S.gp_fit(*args, dtype=dt)
    mu, sd = S.posterior(g, dev(w["Xc"]))
    torch.cuda.synchronize()
    t = TOL[dt]
    assert_close(mu.cpu().numpy(), mu_o, t["mu"], np.max(np.abs(mu_o)), f"{name} mu")
    assert_close(sd.cpu().numpy(), sd_o, t["sd"], np.sqrt(w["signal_var"][obj]), f"{name} sigma")


_ORACLE_POST = {}


@pytest.mark.parametrize("dt", [S.F32, S.F64], ids=["f32", "f64"])
@pytest.mark.parametrize("cfg,m", [(3, 256), (4, 512)], ids=["m256-4waves", "m512-8waves"])
def test_posterior_many_tiles_per_workgroup(cfg, m, dt):
    """The kernels are persistent (one workgroup per slot on the chip, each
    looping over tiles, the inverse-factor stream and the next tile's
    coordinates carried across tiles): 100003 candidates give every workgroup
    several tiles (32 or 64 candidates each) and a ragged last one."""
    n = 100003
    w = wl(cfg, n, m)
    say("posterior many tiles", cfg, "dtype", dt, "m", w["m"], "n", n)
    args = (w["X"], w["Y"][:, 0], w["lengthscale"][0], w["signal_var"][0], w["noise_var"][0], w["prior_mean"][0])
    if (cfg, n, m) not in _ORACLE_POST:
        _ORACLE_POST[(cfg, n, m)] = gp_posterior(gp_fit(*args), w["Xc"].astype(np.float64))
    mu_o, sd_o = _ORACLE_POST[(cfg, n, m)]
    g = S.gp_fit(*args, dtype=dt)
    mu, sd = S.posterior(g, dev(w["Xc"]))
    torch.cuda.synchronize()
    t = TOL[dt]
    assert_close(mu.cpu().numpy(), mu_o, t["mu"], np.max(np.abs(mu_o)), f"many tiles {cfg} mu")
    assert_close(sd.cpu().numpy(), sd_o, t["sd"], np.sqrt(w["signal_var"][0]), f"many tiles {cfg} sigma")


EDGE_SHAPES = [(1, 1, 1, 0.5), (1, 16, 70, 0.5), (31, 16, 63, 0.5), (64, 3, 65, 0.3), (576, 5, 130, 0.4),
               (200, 12, 1, 0.5), (33, 10, 64 * 3 + 1, 0.5)]


@pytest.mark.parametrize("dt", [S.F32, S.F64], ids=["f32", "f64"])
def test_posterior_edge_shapes(dt):
    """Ragged and extreme shapes (m = 1, m = 576 = the maximum, d = 1 and 16 =
    the maximum, n = 1, n not a multiple of the tile), with the conditioning of
    the workloads: kappa(K + tau^2 I) <= 1e4, where the float32 bar applies."""
    rng = np.random.default_rng(5)
    for m, d, n, ls_hi in EDGE_SHAPES:
        say("posterior edge", m, d, n, dt)
        X = rng.random((m, d))
        y = rng.standard_normal(m)
        ls = rng.uniform(0.1, ls_hi, d)
        Xc = rng.random((n, d)).astype(np.float32)
        Xc[0] = X[0]  # a candidate on an observation
        fit = gp_fit(X, y, ls, 1.7, 1e-3, 0.3)
        assert np.linalg.cond(fit["K"]) <= 1e4
        mu_o, sd_o = gp_posterior(fit, Xc.astype(np.float64))
        g = S.gp_fit(X, y, ls, 1.7, 1e-3, 0.3, dtype=dt)
        mu, sd = S.posterior(g, dev(Xc))
        torch.cuda.synchronize()
        t = TOL[dt]
        assert_close(mu.cpu().numpy(), mu_o, t["mu"], np.max(np.abs(mu_o)), f"edge {m},{d},{n} mu")
        assert_close(sd.cpu().numpy(), sd_o, t["sd"], np.sqrt(1.7), f"edge {m},{d},{n} sigma")
    g = S.gp_fit(X, y, ls, 1.7, 1e-3, dtype=dt)
    S.posterior(g, torch.empty((0, d), dtype=torch.float32, device=DEV))  # n = 0 is a no-op
    torch.cuda.synchronize()


def test_posterior_ill_conditioned():
    """kappa(K) ~ 8e4: rounding K* once to float32 already moves mu by 1e-4 of
    its scale, so the float32 path is held to 1e-3 there and the float64 path
    to its usual 1e-10."""
    rng = np.random.default_rng(5)
    for _ in range(4):
        rng.random((1, 1))
    m, d, n = 64, 3, 4096
    X = rng.random((m, d))
    y = rng.standard_normal(m)
    ls = rng.uniform(0.2, 1.5, d)
    Xc = rng.random((n, d)).astype(np.float32)
    fit = gp_fit(X, y, ls, 1.7, 1e-3, 0.3)
    kappa = np.linalg.cond(fit["K"])
    say("posterior ill-conditioned kappa", f"{kappa:.2e}")
    assert kappa > 1e4
    mu_o, sd_o = gp_posterior(fit, Xc.astype(np.float64))
    for dt, rt_mu, rt_sd in [(S.F32, 1e-3, 1e-3), (S.F64, 1e-10, 1e-10)]:
        g = S.gp_fit(X, y, ls, 1.7, 1e-3, 0.3, dtype=dt)
        mu, sd = S.posterior(g, dev(Xc))
        torch.cuda.synchronize()
        assert_close(mu.cpu().numpy(), mu_o, rt_mu, np.max(np.abs(mu_o)), f"ill-conditioned mu {dt}")
        assert_close(sd.cpu().numpy(), sd_o, rt_sd, np.sqrt(1.7), f"ill-conditioned sigma {dt}")


# --------------------------------------------------------------------------- EI / EHVI
@pytest.mark.parametrize("dt", [S.F32, S.F64], ids=["f32", "f64"])
def test_ei_parity(dt):
    rng = np.random.default_rng(7)
    n = 20000
    mu = rng.standard_normal(n) * 2
    sd = np.abs(rng.standard_normal(n)) * 0.5
    sd[:100] = 0.0
    sd[100:200] = 1e-6
    mu[200:300] = 40.0  # deep in the tail
    best = -0.7
    td = torch.float32 if dt == S.F32 else torch.float64
    mu_t, sd_t = dev(mu, td), dev(sd, td)
    want = expected_improvement(as_held(mu, td), as_held(sd, td), best, 1e-4)
    say("ei", dt)
    got = S.acq_ei(mu_t, sd_t, best, 1e-4)
    torch.cuda.synchronize()
    assert_close(got.cpu().numpy(), want, TOL[dt]["acq"], np.max(want), "ei")


def _ehvi_case(p, size, seed):
    rng = np.random.default_rng(seed)
    Y = rng.standard_normal((size, p))
    if p >= 2:
        Y[:, 1] = -0.9 * Y[:, 0] + 0.2 * Y[:, 1]
    ref = Y.max(axis=0) + 0.1 * (Y.max(axis=0) - Y.min(axis=0))
    return Y, ref


@pytest.mark.parametrize("dt", [S.F32, S.F64], ids=["f32", "f64"])
@pytest.mark.parametrize("p,size", [(1, 10), (2, 1), (2, 40), (3, 25), (2, 0), (3, 0)])
def test_ehvi_parity_shared_inputs(p, size, dt):
    Y, ref = _ehvi_case(p, max(size, 1), 100 + p * 7 + size)
    if size == 0:
        Y = np.zeros((0, p))
        ref = np.ones(p)
    rng = np.random.default_rng(3)
    n = 3000
    mu = rng.standard_normal((n, p)) * 1.2
    sd = np.abs(rng.standard_normal((n, p))) * 0.4
    sd[:20] = 0.0
    mu[20:40] = ref + 5.0
    td = torch.float32 if dt == S.F32 else torch.float64
    mus = [dev(mu[:, j], td) for j in range(p)]
    sds = [dev(sd[:, j], td) for j in range(p)]
    mu_c, sd_c = as_held(mu, td), as_held(sd, td)
    want = oracle_ehvi(mu_c, sd_c, nondominated(Y, ref) if len(Y) else np.zeros((0, p)), ref)
    say("ehvi", p, size, dt)
    got = S.acq_ehvi(mus, sds, Y, ref)
    torch.cuda.synchronize()
    assert_close(got.cpu().numpy(), want, TOL[dt]["acq"], max(np.max(want), 1e-300), f"ehvi p={p}")


@pytest.mark.parametrize("dt", [S.F32, S.F64], ids=["f32", "f64"])
def test_ehvi3_parity_tied_coordinates(dt):
    """Three objectives whose front shares coordinate values on every axis
    (values on a quarter grid): merged axis coordinates, boxes spanning
    several of them, candidates exactly on box edges."""
    rng = np.random.default_rng(77)
    Y = np.round(rng.standard_normal((40, 3)) * 4) / 4
    Y[:, 2] = np.round((-0.6 * Y[:, 0] - 0.5 * Y[:, 1] + 0.3 * rng.standard_normal(40)) * 4) / 4
    ref = Y.max(axis=0) + 0.5
    n = 4096 + 3
    mu = np.round(rng.standard_normal((n, 3)) * 4) / 4
    sd = np.abs(rng.standard_normal((n, 3))) * 0.3
    sd[:64] = 0.0
    td = torch.float32 if dt == S.F32 else torch.float64
    mus = [dev(mu[:, j], td) for j in range(3)]
    sds = [dev(sd[:, j], td) for j in range(3)]
    mu_c, sd_c = as_held(mu, td), as_held(sd, td)
    P = nondominated(Y, ref)
    want = oracle_ehvi(mu_c, sd_c, P, ref)
    say("ehvi3 tied coordinates", dt, len(P))
    got = S.acq_ehvi(mus, sds, Y, ref)
    torch.cuda.synchronize()
    assert_close(got.cpu().numpy(), want, TOL[dt]["acq"], np.max(want), "ehvi p=3 ties")


@pytest.mark.parametrize("cfg", [3, 4])
def test_ehvi_parity_workload_front(cfg):
    w = wl(cfg, 2048)
    P = nondominated(w["Y"], w["ref"])
    rng = np.random.default_rng(cfg)
    p = w["p"]
    mu = w["Y"][rng.integers(0, w["m"], 2048)] + 0.3 * rng.standard_normal((2048, p))
    sd = rng.uniform(0.01, 1.0, (2048, p))
    mus = [dev(mu[:, j]) for j in range(p)]
    sds = [dev(sd[:, j]) for j in range(p)]
    mu_c, sd_c = as_held(mu, torch.float32), as_held(sd, torch.float32)
    want = oracle_ehvi(mu_c, sd_c, P, w["ref"])
    say("ehvi workload front", cfg, len(P))
    got = S.acq_ehvi(mus, sds, w["Y"], w["ref"])
    torch.cuda.synchronize()
    assert_close(got.cpu().numpy(), want, 1e-3, np.max(want), f"ehvi cfg{cfg}")


# --------------------------------------------------------------------------- forest
def _forest(fd, d):
    return S.forest_create(fd["feature"], fd["threshold"], fd["left"], fd["right"], fd["leaf_q16"],
                           fd["tree_offset"], d)


def test_forest_hand_traced(golden_dir):
    import json
    import os
    with open(os.path.join(golden_dir, "hand_trees.json")) as fh:
        g = json.load(fh)
    f = S.forest_create(g["feature"], np.array(g["threshold"], np.float32), g["left"], g["right"], g["leaf_q16"],
                        g["tree_offset"], g["d"])
    X = dev(np.array(g["X"], np.float32))
    for delta, key in [(0.5, "mask_delta_0.5"), (0.6, "mask_delta_0.6")]:
        say("forest hand", delta)
        votes, mask, leaves = S.rf_feasibility(f, X, delta, leaf_idx=True)
        torch.cuda.synchronize()
        assert leaves.cpu().numpy().tolist() == g["leaves"]
        assert votes.cpu().numpy().tolist() == g["votes"]
        assert mask.cpu().numpy().tolist() == g[key]


@pytest.mark.parametrize("cfg", [1, 2, 4])
def test_forest_bitexact(cfg):
    w = wl(cfg, 20000 + cfg)
    fd = w["forest"]
    Xc = w["Xc"].copy()
    Xc[:7, 0] = np.nan
    f = _forest(fd, w["d"])
    say("forest", cfg, "trees", len(fd["tree_offset"]) - 1, "nodes", fd["tree_offset"][-1])
    for delta in (0.25, 0.5, 0.55, 0.75):
        votes, mask, leaves = S.rf_feasibility(f, dev(Xc), delta, leaf_idx=True)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(leaves.cpu().numpy(), forest_apply(fd, Xc))
        v_o = forest_votes(fd, Xc)
        np.testing.assert_array_equal(votes.cpu().numpy(), v_o)
        np.testing.assert_array_equal(mask.cpu().numpy(), feasibility_mask(v_o, delta, len(fd["tree_offset"]) - 1))


def _grid_forest(rng, depths, d, grids, full=False, p0=0.0):
    """Random trees whose thresholds come from per-feature value grids (so
    candidates can sit exactly on them), one tree per entry of depths; with
    full=True each tree is complete to its depth; p0 is the share of splits
    forced onto feature 0."""
    feat, thr, left, right, q16, off = [], [], [], [], [], [0]
    for depth in depths:
        nodes = []

        def grow(level):
            me = len(nodes)
            nodes.append(None)
            if level == depth or (not full and level > 0 and rng.random() < 0.25):
                nodes[me] = (-1, 0.0, -1, -1, int(rng.integers(0, 65537)))
                return me
            k = 0 if rng.random() < p0 else int(rng.integers(0, d))
            t = grids[k][int(rng.integers(0, len(grids[k])))]
            lo = grow(level + 1)
            hi = grow(level + 1)
            nodes[me] = (k, t, lo, hi, 0)
            return me

        grow(0)
        for k, t, lo, hi, q in nodes:
            feat.append(max(k, 0))
            thr.append(t)
            left.append(lo)
            right.append(hi)
            q16.append(q)
        off.append(off[-1] + len(nodes))
    return dict(feature=np.array(feat, np.int32), threshold=np.array(thr, np.float32),
                left=np.array(left, np.int32), right=np.array(right, np.int32),
                leaf_q16=np.array(q16, np.int32), tree_offset=np.array(off, np.int64))


def _near_candidates(rng, n, d, grids):
    """Candidates on the grid values, one float32 step either side of them,
    at +-0, +-inf and NaN, and uniform ones."""
    X = rng.uniform(-2, 2, (n, d)).astype(np.float32)
    for k in range(d):
        g = np.asarray(grids[k], np.float32)
        pick = g[rng.integers(0, len(g), n)]
        side = rng.integers(0, 4, n)
        near = np.where(side == 0, pick, np.where(side == 1, np.nextafter(pick, np.float32(np.inf)),
                                                  np.where(side == 2, np.nextafter(pick, np.float32(-np.inf)), X[:, k])))
        X[:, k] = near
    special = np.array([0.0, -0.0, np.inf, -np.inf, np.nan], np.float32)
    sel = rng.random((n, d)) < 0.05
    X[sel] = special[rng.integers(0, len(special), sel.sum())]
    return X


def _check_forest(fd, d, X, what):
    f = _forest(fd, d)
    T = len(fd["tree_offset"]) - 1
    for delta in (0.3, 0.6):
        say(what, "n", len(X), "trees", T, "nodes", fd["tree_offset"][-1], "delta", delta)
        votes, mask, leaves = S.rf_feasibility(f, dev(X), delta, leaf_idx=True)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(leaves.cpu().numpy(), forest_apply(fd, X))
        v_o = forest_votes(fd, X)
        np.testing.assert_array_equal(votes.cpu().numpy(), v_o)
        np.testing.assert_array_equal(mask.cpu().numpy(), feasibility_mask(v_o, delta, T))


def _grids(rng, d, counts):
    base = [0.0, -0.0, np.inf, -np.inf, -1.5, 1e-30, -1e-30]
    out = []
    for k in range(d):
        extra = np.unique(rng.uniform(-2, 2, 4 * counts[k]).astype(np.float32))
        vals = np.unique(np.concatenate([np.array(base, np.float32), extra]))  # -0.0 == 0.0: one entry
        out.append(vals[: counts[k]] if counts[k] < len(vals) else vals)
    return out


@pytest.mark.parametrize("top", [254, 255])
def test_forest_ties_and_special_values(top):
    """Every branch matches the oracle's float32 comparison bit for bit with
    candidates on the thresholds and one float32 step either side of them,
    thresholds and candidates at +-0, +-inf, NaN candidates, all sixteen
    feature slots, and one feature with a few hundred distinct thresholds."""
    rng = np.random.default_rng(top)
    d = 16
    counts = [top] + [int(c) for c in rng.integers(1, 40, d - 1)]
    grids = _grids(rng, d, counts)
    fd = _grid_forest(rng, [9] * 40, d, grids, p0=0.5)
    k = np.where((fd["left"] >= 0) & (fd["feature"] == 0))[0]
    fd["threshold"][k[: len(grids[0])]] = grids[0]  # every value of feature 0's grid on some node
    z = k[fd["threshold"][k] == 0]
    fd["threshold"][z[::2]] = -0.0  # signed zeros: one threshold value
    assert len(np.unique(fd["threshold"][(fd["left"] >= 0) & (fd["feature"] == 0)])) == top
    assert fd["tree_offset"][-1] < 8192
    _check_forest(fd, d, _near_candidates(rng, 20000 + 37, d, grids), f"forest {top} thresholds")


def test_forest_largest_tree_and_two_chunks():
    """A complete tree of 8191 nodes (the largest one chunk holds) and one of
    4095 nodes land in two chunks of one forest, one launch each, with the
    votes carried between them."""
    rng = np.random.default_rng(7)
    d = 5
    grids = _grids(rng, d, [30, 20, 10, 5, 3])
    fd = _grid_forest(rng, [12, 11], d, grids, full=True)
    assert np.diff(fd["tree_offset"]).tolist() == [8191, 4095]
    _check_forest(fd, d, _near_candidates(rng, 9000 + 5, d, grids), "forest 8191 + 4095 nodes")


# --------------------------------------------------------------------------- top-q
@pytest.mark.parametrize("dt", [S.F32, S.F64], ids=["f32", "f64"])
def test_topq_bitexact_shared_scores(dt):
    rng = np.random.default_rng(11)
    td = torch.float32 if dt == S.F32 else torch.float64
    npd = np.float32 if dt == S.F32 else np.float64
    for n, q in [(0, 1), (1, 1), (5, 8), (4096, 4), (4097, 64), (262144 + 3, 4), (1048576, 8), (3000000, 16)]:
        say("topq", n, q, dt)
        score = rng.integers(-50, 50, n).astype(npd)  # many ties
        score[rng.random(n) < 0.01] = np.nan
        if n > 10:
            score[3] = -0.0
            score[4] = 0.0
            score[5] = np.inf
            score[6] = -np.inf
        mask = (rng.random(n) < 0.8).astype(np.uint8)
        idx, val, nv = S.suggest_topq(dev(score, td), dev(mask, torch.uint8), q)
        torch.cuda.synchronize()
        want_idx, want_val, want_nv = top_q(score, mask, q)
        assert idx.cpu().numpy().tolist() == want_idx.tolist()
        assert int(nv.cpu().numpy()[0]) == want_nv
        np.testing.assert_array_equal(val.cpu().numpy().astype(np.float64), want_val)


def test_topq_no_mask_and_all_masked():
    score = dev(np.arange(100, dtype=np.float32))
    idx, _, nv = S.suggest_topq(score, None, 3)
    torch.cuda.synchronize()
    assert idx.cpu().tolist() == [99, 98, 97] and int(nv.cpu()[0]) == 100
    idx, val, nv = S.suggest_topq(score, dev(np.zeros(100, np.uint8), torch.uint8), 3)
    torch.cuda.synchronize()
    assert idx.cpu().tolist() == [-1, -1, -1] and int(nv.cpu()[0]) == 0 and torch.isnan(val).all()


# --------------------------------------------------------------------------- whole pass
def _check_pool(w, b, ref, dt):
    p = w["p"]
    t = TOL[dt]
    for j in range(p):
        assert_close(b.mu[j].cpu().numpy(), ref["mu"][:, j], t["mu"], np.max(np.abs(ref["mu"][:, j])), f"mu{j}")
        assert_close(b.sigma[j].cpu().numpy(), ref["sigma"][:, j], t["sd"], 1.0, f"sigma{j}")
    assert_close(b.acq.cpu().numpy(), ref["acq"], t["acq"], np.max(ref["acq"]), "acq")
    np.testing.assert_array_equal(b.votes.cpu().numpy(), ref["votes"])
    np.testing.assert_array_equal(b.mask.cpu().numpy(), ref["mask"])
    assert int(b.n_valid.cpu()[0]) == ref["n_valid"]
    # Indices: exact where the oracle's ranking is decided beyond the
    # tolerance; otherwise every pick must score within tolerance of the
    # oracle's q-th best.
    q = w["q"]
    acq_o = np.where(ref["mask"] != 0, ref["acq"], -np.inf)
    order = np.lexsort((np.arange(len(acq_o)), -acq_o))
    tol = t["acq"] * np.max(ref["acq"])
    gap = acq_o[order[q - 1]] - acq_o[order[q]] if len(order) > q else np.inf
    got = b.idx.cpu().numpy()
    if gap > 2 * tol:
        assert set(got.tolist()) == set(order[:q].tolist())
    for i in got:
        assert ref["mask"][i] == 1 and acq_o[i] >= acq_o[order[q - 1]] - 2 * tol


@pytest.mark.parametrize("cfg,n,dt", [(1, 4096, S.F32), (1, 4096, S.F64), (2, 16384, S.F32), (3, 16384, S.F32),
                                      (4, 4096, S.F32), (4, 2048, S.F64)])
def test_score_pool_end_to_end(cfg, n, dt):
    w = wl(cfg, n)
    ref = oracle_score_pool(w)
    gps = [S.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], w["signal_var"][j], w["noise_var"][j],
                    w["prior_mean"][j], dtype=dt) for j in range(w["p"])]
    f = _forest(w["forest"], w["d"])
    say("score_pool", cfg, n, dt)
    b = S.score_pool(gps, f, dev(w["Xc"]), w["q"], best_y=w["best_y"], xi=w["xi"], Y_obs=w["Y"],
                     ref=w.get("ref"), delta=w["delta"])
    torch.cuda.synchronize()
    _check_pool(w, b, ref, dt)


def test_full_size_two_objective_pool():
    """The measured workload at its real size (m = 256, n = 262144, two
    objectives), in the launch configuration the bench times: mu, sigma and
    EHVI of every candidate against the oracle one by one, votes and mask everywhere,
    and the top-q picks against the oracle's ranking of the whole pool (exact
    where the oracle's cut is clear, within the bar at a near tie)."""
    w = wl(3, None)
    n = len(w["Xc"])
    gps = [S.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], 1.0, w["noise_var"][j], dtype=S.F32)
           for j in range(2)]
    f = _forest(w["forest"], w["d"])
    say("full size cfg3", n)
    Xd = dev(w["Xc"])
    b = S.score_pool(gps, f, Xd, w["q"], Y_obs=w["Y"], ref=w["ref"], delta=w["delta"])
    torch.cuda.synchronize()
    mu_o = np.empty((n, 2))
    sd_o = np.empty((n, 2))
    X64 = w["Xc"].astype(np.float64)
    for j in range(2):
        fit = gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], 1.0, w["noise_var"][j])
        mu_o[:, j], sd_o[:, j] = gp_posterior(fit, X64)
    for j in range(2):
        assert_close(b.mu[j].cpu().numpy(), mu_o[:, j], 1e-4, np.max(np.abs(mu_o[:, j])), f"mu{j}")
        assert_close(b.sigma[j].cpu().numpy(), sd_o[:, j], 1e-3, 1.0, f"sigma{j}")
    e_o = oracle_ehvi(mu_o, sd_o, nondominated(w["Y"], w["ref"]), w["ref"])
    acq = b.acq.cpu().numpy()
    assert_close(acq, e_o, 1e-3, np.max(e_o), "ehvi")
    v_o = forest_votes(w["forest"], w["Xc"])
    np.testing.assert_array_equal(b.votes.cpu().numpy(), v_o)
    mask_o = feasibility_mask(v_o, w["delta"], 64)
    np.testing.assert_array_equal(b.mask.cpu().numpy(), mask_o)
    check_topq(b.idx.cpu().numpy(), b.n_valid.cpu()[0], e_o, mask_o, w["q"], 1e-3)


def test_full_size_three_objective_pool():
    """The three-objective workload at its real size (m = 512, n = 2^20, d = 12:
    the eight-wave posterior, the per-column EHVI, 128 trees of depth 12), in
    the launch configuration the bench times: mu, sigma, EHVI, votes and the
    mask on a seeded sample of candidates against the oracle one by one, and
    the picks eligible, distinct and in order of the library's own scores."""
    w = wl(4, None)
    n, p = len(w["Xc"]), 3
    gps = [S.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], 1.0, w["noise_var"][j], dtype=S.F32)
           for j in range(p)]
    f = _forest(w["forest"], w["d"])
    say("full size cfg4", n)
    b = S.score_pool(gps, f, dev(w["Xc"]), w["q"], Y_obs=w["Y"], ref=w["ref"], delta=w["delta"])
    torch.cuda.synchronize()
    rng = np.random.default_rng(1)
    sample = np.unique(np.concatenate([rng.integers(0, n, 3000), np.arange(n - 64, n)]))
    Xs = w["Xc"][sample].astype(np.float64)
    mu_o = np.empty((len(sample), p))
    sd_o = np.empty((len(sample), p))
    for j in range(p):
        fit = gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], 1.0, w["noise_var"][j])
        mu_o[:, j], sd_o[:, j] = gp_posterior(fit, Xs)
        assert_close(b.mu[j].cpu().numpy()[sample], mu_o[:, j], 1e-4, np.max(np.abs(mu_o[:, j])), f"mu{j}")
        assert_close(b.sigma[j].cpu().numpy()[sample], sd_o[:, j], 1e-3, 1.0, f"sigma{j}")
    e_o = oracle_ehvi(mu_o, sd_o, nondominated(w["Y"], w["ref"]), w["ref"])
    acq = b.acq.cpu().numpy()
    assert_close(acq[sample], e_o, 1e-3, np.max(e_o), "ehvi")
    v_o = forest_votes(w["forest"], w["Xc"][sample])
    np.testing.assert_array_equal(b.votes.cpu().numpy()[sample], v_o)
    mask_o = feasibility_mask(v_o, w["delta"], len(w["forest"]["tree_offset"]) - 1)
    mask_g = b.mask.cpu().numpy()
    np.testing.assert_array_equal(mask_g[sample], mask_o)
    got = b.idx.cpu().numpy()
    assert len(set(got.tolist())) == len(got) and np.all(mask_g[got] == 1)
    assert np.all(np.diff(acq[got]) <= 0) and acq[got[-1]] >= np.max(np.where(mask_g != 0, acq, -np.inf)[
        np.setdiff1d(np.arange(n), got)])


def test_repeat_runs_bit_identical():
    w = wl(3, 16384)
    gps = [S.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], 1.0, w["noise_var"][j]) for j in range(2)]
    f = _forest(w["forest"], w["d"])
    Xd = dev(w["Xc"])
    outs = []
    for _ in range(3):
        say("repeat")
        b = S.score_pool(gps, f, Xd, w["q"], Y_obs=w["Y"], ref=w["ref"], delta=w["delta"])
        torch.cuda.synchronize()
        outs.append([t.cpu().numpy().copy() for t in (b.mu, b.sigma, b.acq, b.votes, b.mask, b.idx)])
    for o in outs[1:]:
        for a, c in zip(outs[0], o):
            np.testing.assert_array_equal(a, c)


# --------------------------------------------------------------------------- believer
# (n, m, q): the oracle's own greedy sequence is decided (best clear of the
# runner-up by more than twice the bar) at every step of these pools, so the
# whole sequence must agree.  m = 40 and 200 run the four-wave posterior;
# m = 512 (the three-objective workload's observations, two objectives, eight
# picks) runs the eight-wave posterior that keeps V and row updates over
# 512 .. 518 rows, on a pool of 641 tiles of 64 (several per workgroup) with a
# ragged tail.
@pytest.mark.parametrize("n,m,q", [(2048 + 7, 40, 8), (16384, 200, 6), (40960 + 13, None, 8)])
def test_believer_sequence(n, m, q):
    w = wl(5, n, m)
    p = 2
    gps = [S.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], w["signal_var"][j], w["noise_var"][j],
                    w["prior_mean"][j]) for j in range(p)]
    f = _forest(w["forest"], w["d"])
    say("believer", n, w["m"], q)
    mu_g = torch.empty((p, n), dtype=torch.float32, device=DEV)
    sd_g = torch.empty((p, n), dtype=torch.float32, device=DEV)
    picks, acq_g = S.suggest_kb(gps, f, dev(w["Xc"]), q, w["Y"], w["ref"], delta=w["delta"], mu_out=mu_g,
                                sigma_out=sd_g)
    torch.cuda.synchronize()
    assert len(picks) == q and len(set(picks.tolist())) == q
    mask = feasibility_mask(forest_votes(w["forest"], w["Xc"]), w["delta"], len(w["forest"]["tree_offset"]) - 1)
    _, mu_o, sd_o = check_believer(w, q, picks, acq_g, mask, min_steps=q)
    # the whole sequence agreed: the last round's posterior is the oracle's
    # refit on the observations plus q - 1 fantasies, on every candidate
    for j in range(p):
        assert_close(mu_g[j].cpu().numpy(), mu_o[:, j], 1e-4, np.max(np.abs(mu_o[:, j])), f"mu{j}")
        assert_close(sd_g[j].cpu().numpy(), sd_o[:, j], 1e-3, np.sqrt(w["signal_var"][j]), f"sigma{j}")


def test_believer_shortfall_and_workspace():
    w = wl(5, 300, 40)
    gps = [S.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], 1.0, w["noise_var"][j]) for j in range(2)]
    Xc = dev(w["Xc"])
    nbytes = S.suggest_kb_workspace(gps, 300, 4)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    say("believer workspace", nbytes)
    p1, a1 = S.suggest_kb(gps, None, Xc, 4, w["Y"], w["ref"], workspace=ws)
    p2, a2 = S.suggest_kb(gps, None, Xc, 4, w["Y"], w["ref"])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(p1, p2)
    np.testing.assert_array_equal(a1, a2)
    # every candidate infeasible: no pick
    f = _forest(w["forest"], w["d"])
    p3, _ = S.suggest_kb(gps, f, Xc, 4, w["Y"], w["ref"], delta=1.0)
    mask = feasibility_mask(forest_votes(w["forest"], w["Xc"]), 1.0, len(w["forest"]["tree_offset"]) - 1)
    assert len(p3) == min(4, int(mask.sum()))


@pytest.mark.parametrize("cfg,T,depth", [(1, 16, 6), (2, 24, 10)])
def test_trained_forest_votes_bitexact(cfg, T, depth):
    from oracle.forest_train import train_forest, voting_format
    w = wl(cfg, 8192 + 11)
    say("forest train + mask", cfg, T, depth)
    f = S.forest_train_create(w["X_draws"], w["feasible_draws"], T, depth, seed=99)
    votes, mask, _ = S.rf_feasibility(f, dev(w["Xc"]), w["delta"])
    torch.cuda.synchronize()
    fo = voting_format(train_forest(w["X_draws"], w["feasible_draws"], T, depth, seed=99))
    want = forest_votes(fo, w["Xc"])
    np.testing.assert_array_equal(votes.cpu().numpy(), want)
    np.testing.assert_array_equal(mask.cpu().numpy(), feasibility_mask(want, w["delta"], T))


def test_oversized_pool_is_rejected():
    """The fused pass and the believer pack a 32-bit inverted index into their
    top-q keys: pools of 2^31 or more candidates are refused before any device
    work (the pointers below are never touched)."""
    from paper_2408_04323_amd._native import lib
    import ctypes as C
    w = wl(3, 1024)
    gps = [S.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], 1.0, w["noise_var"][j]) for j in range(2)]
    hs = (C.c_void_p * 2)(*[g.handle.value for g in gps])
    fake = C.c_void_p(256)
    Y = np.ascontiguousarray(w["Y"], dtype=np.float64)
    r = np.ascontiguousarray(w["ref"], dtype=np.float64)
    pY = Y.ctypes.data_as(C.POINTER(C.c_double))
    pr = r.ctypes.data_as(C.POINTER(C.c_double))
    for n in (1 << 31, 1 << 32):
        say("oversized", n)
        rc = lib().scoot_score_pool_ex(hs, 2, None, None, fake, n, 0.0, 1e-4, pY, len(Y), pr, 0.5, 4, fake, fake,
                                       fake, fake, fake, fake, fake, fake, None)
        assert rc == -1
        b = C.c_uint64(0)
        assert lib().scoot_suggest_kb_workspace(hs, 2, n, 4, C.byref(b)) == -1
    assert lib().scoot_suggest_kb_workspace(hs, 2, (1 << 31) - 1, 4, C.byref(b)) == 0
