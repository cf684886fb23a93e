"""GPU parity of candidate generation: the Sobol pool on the space's grids
and the known-constraint mask are bit-exact against the oracle (integer and
exactly rounded work); the mask folded into the scoring calls is bit-exact
too, and their picks are checked on it."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2408_04323_amd as S  # noqa: E402
from oracle.forest import feasibility_mask, forest_votes  # noqa: E402
from oracle.pipeline import score_pool as oracle_score_pool  # noqa: E402
from oracle.sobol import known_constraints_mask, sobol_pool as oracle_pool  # noqa: E402
from tests.oracle_checks import check_believer, check_topq  # noqa: E402
from workloads import CONFIGS, levels, make_workload, sobol_table, space_constraints, vllm_space  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def _space(name):
    if name == "vllm":
        sp = vllm_space()
        return sp["levels"], sp["A"], sp["b"]
    if name.startswith("cfg"):
        c = CONFIGS[int(name[3:])]
        A, b = space_constraints(c)
        return levels(c), A, b
    d = int(name[1:])
    rng = np.random.default_rng(d)
    lv = rng.choice([0, 1, 2, 3, 7, 64, 8129], size=d).tolist()
    A = rng.choice([-1.0, 0.0, 1.0, 0.375], size=(2, d))
    return lv, A, np.array([0.0, 0.5])


def _forest(fd, d):
    return S.forest_create(fd["feature"], fd["threshold"], fd["left"], fd["right"], fd["leaf_q16"],
                           fd["tree_offset"], d)


def _oracle_rows(poly, vinit, lv, rows, skip):
    """Pool rows one by one (each Sobol point stands on its own)."""
    return np.vstack([oracle_pool(poly, vinit, lv, 1, skip=skip + int(i)) for i in rows])


# (space, n, skip): runs of 16 cut by the start and the end, one and several
# blocks, every block width (d = 1 .. 16), the last points of the 2^32 period.
CASES = [("d1", 5000, 0), ("d1", 17, 3), ("d3", 4099, 13), ("cfg1", 4096, 0), ("cfg4", 5003, 1),
         ("vllm", 4111, 16), ("d16", 3000, 1000003), ("d5", 1000, (1 << 32) - 1000), ("cfg4", 1, 7),
         ("d16", 15, 1), ("d7", 0, 5)]


@pytest.mark.parametrize("space,n,skip", CASES, ids=[f"{c[0]}-n{c[1]}-s{c[2]}" for c in CASES])
def test_sobol_pool_bitexact(space, n, skip):
    lv, A, b = _space(space)
    d = len(lv)
    poly, vinit = sobol_table(d)
    say("sobol", space, n, skip)
    Xc, known = S.sobol_pool(poly, vinit, lv, n, skip=skip, A=A, b=b, device=DEV)
    torch.cuda.synchronize()
    want = oracle_pool(poly, vinit, lv, n, skip=skip)
    got = Xc.cpu().numpy()
    assert got.shape == (n, d)
    np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32))
    np.testing.assert_array_equal(known.cpu().numpy(), known_constraints_mask(want, A, b))


def test_sobol_pool_without_constraints_and_into_given_buffers():
    lv, _, _ = _space("cfg3")
    poly, vinit = sobol_table(len(lv))
    n = 2000
    out = torch.full((n, len(lv)), -7.0, device=DEV)
    known = torch.full((n,), 9, dtype=torch.uint8, device=DEV)
    say("sobol given buffers")
    S.sobol_pool(poly, vinit, lv, n, skip=5, out=out, known=known)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy(), oracle_pool(poly, vinit, lv, n, skip=5))
    assert np.all(known.cpu().numpy() == 1)  # no rows: every candidate admissible
    Xc, k2 = S.sobol_pool(poly, vinit, lv, n, skip=5)
    torch.cuda.synchronize()
    assert k2 is None
    np.testing.assert_array_equal(Xc.cpu().numpy(), out.cpu().numpy())


def test_sobol_pool_full_size():
    """The three-objective space at n = 2^20: sampled rows and their mask
    entries against the oracle point by point, and the exact balance of every
    boolean over the power-of-two pool."""
    c = CONFIGS[4]
    lv = levels(c)
    A, b = space_constraints(c)
    d = len(lv)
    n = c["n"]
    poly, vinit = sobol_table(d)
    say("sobol full size", n, d)
    Xc, known = S.sobol_pool(poly, vinit, lv, n, A=A, b=b, device=DEV)
    torch.cuda.synchronize()
    X = Xc.cpu().numpy()
    rng = np.random.default_rng(4)
    per_block = (256 // d) * 16
    edges = np.concatenate([np.arange(k * per_block - 3, k * per_block + 3) for k in (1, 2, 777, n // per_block)])
    rows = np.unique(np.concatenate([rng.integers(0, n, 300), np.arange(40), np.arange(n - 40, n), edges]))
    rows = rows[(rows >= 0) & (rows < n)]
    Xo = _oracle_rows(poly, vinit, lv, rows, 0)
    np.testing.assert_array_equal(X[rows], Xo)
    np.testing.assert_array_equal(known.cpu().numpy()[rows], known_constraints_mask(Xo, A, b))
    for j, L in enumerate(lv):
        if L == 1:
            assert np.count_nonzero(X[:, j]) == n // 2
        elif L >= 2:
            k = X[:, j].astype(np.float64) * (L - 1)
            assert np.all(np.abs(k - np.rint(k)) < 1e-5) and k.min() == 0 and np.rint(k).max() == L - 1


def test_known_constraints_standalone():
    """Any pool (the uniform workload pool, with NaN and signed-zero rows): bit-exact."""
    w = make_workload(4, n=6000, with_forest=False)
    A, b = space_constraints(w["config"])
    X = w["Xc"].copy()
    X[5, :] = np.nan
    X[6, :] = -0.0
    X[7, :] = 0.0
    say("known constraints standalone")
    Xd = torch.as_tensor(X).to(DEV)
    got = S.known_constraints(Xd, A, b)
    torch.cuda.synchronize()
    want = known_constraints_mask(X, A, b)
    np.testing.assert_array_equal(got.cpu().numpy(), want)
    assert want[5] == 0 and 0.1 < want.mean() < 0.9
    none = S.known_constraints(Xd, None, None)
    torch.cuda.synchronize()
    assert np.all(none.cpu().numpy() == 1)


def _sobol_workload(cfg, n, m=None):
    w = make_workload(cfg, n=16, m=m)
    c = w["config"]
    lv = levels(c)
    A, b = space_constraints(c)
    poly, vinit = sobol_table(len(lv))
    Xc, known = S.sobol_pool(poly, vinit, lv, n, skip=1, A=A, b=b, device=DEV)
    torch.cuda.synchronize()
    # the oracle's side is generated by the oracle; the two pools are the same
    w["Xc"] = oracle_pool(poly, vinit, lv, n, skip=1)
    kn = known_constraints_mask(w["Xc"], A, b)
    np.testing.assert_array_equal(Xc.cpu().numpy(), w["Xc"])
    np.testing.assert_array_equal(known.cpu().numpy(), kn)
    return w, Xc, known, kn


def test_score_pool_with_known_mask():
    w, Xd, known, kn = _sobol_workload(3, 20000)
    gps = [S.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], 1.0, w["noise_var"][j]) for j in range(2)]
    f = _forest(w["forest"], w["d"])
    say("score pool known")
    bk = S.score_pool(gps, f, Xd, w["q"], Y_obs=w["Y"], ref=w["ref"], delta=w["delta"], known=known)
    torch.cuda.synchronize()
    mask_o = feasibility_mask(forest_votes(w["forest"], w["Xc"]), w["delta"], 64) & kn
    np.testing.assert_array_equal(bk.mask.cpu().numpy(), mask_o)
    ref = oracle_score_pool(w)
    check_topq(bk.idx.cpu().numpy(), bk.n_valid.cpu()[0], ref["acq"], mask_o, w["q"], 1e-3)
    # without a forest the mask is the known mask itself
    b0 = S.score_pool(gps, None, Xd, w["q"], Y_obs=w["Y"], ref=w["ref"], known=known)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(b0.mask.cpu().numpy(), kn)


def test_suggest_mace_with_known_mask():
    w, Xd, known, kn = _sobol_workload(2, 20000)
    gp = S.gp_fit(w["X"], w["Y"][:, 0], w["lengthscale"][0], 1.0, w["noise_var"][0])
    f = _forest(w["forest"], w["d"])
    say("mace known")
    b = S.suggest_mace(gp, f, Xd, 4, w["best_y"], S.ucb_beta(3), seed=11, delta=w["delta"], known=known)
    torch.cuda.synchronize()
    mask_o = feasibility_mask(forest_votes(w["forest"], w["Xc"]), w["delta"], 64) & kn
    np.testing.assert_array_equal(b.mask.cpu().numpy(), mask_o)
    front = b.front.cpu().numpy()
    assert np.all(mask_o[front != 0] == 1) and front.sum() >= 1
    assert all(front[i] == 1 for i in b.idx.cpu().numpy() if i >= 0)


def test_suggest_kb_with_known_mask():
    w, Xd, known, kn = _sobol_workload(5, 2055, m=40)
    gps = [S.gp_fit(w["X"], w["Y"][:, j], w["lengthscale"][j], w["signal_var"][j], w["noise_var"][j],
                    w["prior_mean"][j]) for j in range(2)]
    f = _forest(w["forest"], w["d"])
    q = 4
    say("believer known")
    picks, acq_g = S.suggest_kb(gps, f, Xd, q, w["Y"], w["ref"], delta=w["delta"], known=known)
    torch.cuda.synchronize()
    mask = feasibility_mask(forest_votes(w["forest"], w["Xc"]), w["delta"], 128) & kn
    assert len(picks) == q and all(mask[i] for i in picks)
    check_believer(w, q, picks, acq_g, mask)
