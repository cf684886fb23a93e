"""Seeded generators shaped like LLM-engine parameter search spaces.

The paper tunes engine knobs of four kinds, continuous, integer, enumerated
and boolean (Table 1), over a space of more than 1e11 points.  The real engines,
request traces and stress tests are not available here, so every input is
synthetic:

* a configuration is a vector in [0, 1]^d, dimensions ordered
  [continuous..., integer..., boolean...]; an integer dimension with L levels is
  rounded to the grid k / (L - 1) (round half to even), a boolean one to
  x >= 0.5; rounding is done in float64, the pool is then stored as float32;
* SLO values come from smooth seeded functions (sines for the tiny case,
  random Fourier features for the others) plus Gaussian noise, standardised
  over the feasible observations; all objectives are minimised;
* hidden constraints ("crashes") come from a seeded region: a half-plane for
  the tiny case, the intersection of two random half-spaces covering 30% of
  the space for the others;
* observations are drawn uniformly until m feasible ones are collected; the GP
  sees only the feasible ones, the random forest is trained on every draw with
  label 1 = feasible, 0 = crashed (scikit-learn, the paper's own tool);
* the forest is exported as flat node arrays: thresholds rounded DOWN to
  float32 (so that x <= t agrees with the float64 threshold for every float32
  x), leaf values as Q16 integers round(v * 65536).

Seeds: numpy SeedSequence([MASTER_SEED, config]) spawns independent streams
for observations, pool, objective, noise, hyperparameters, hidden region,
forest and a spare.
"""
import numpy as np

MASTER_SEED = 240804323

# Shapes of the five workloads.  "rho" is the correlation between objectives
# of the random-Fourier-feature functions, chosen per workload so that the
# observed Pareto front has roughly the size the workload names (about 30
# points for two objectives at m = 256, about 60 for three at m = 512).
CONFIGS = {
    1: dict(name="tiny-ei", d_cont=3, d_int=3, int_levels=16, d_bool=2, m=32, n=4096, p=1,
            trees=16, depth=6, q=1, noise=1e-4, objective="sines", hidden="halfplane"),
    2: dict(name="mid-ei", d_cont=4, d_int=4, int_levels=32, d_bool=2, m=128, n=262144, p=1,
            trees=64, depth=10, q=4, noise=1e-3, objective="rff", hidden="hyperplane_pair"),
    3: dict(name="two-objective-ehvi", d_cont=4, d_int=4, int_levels=32, d_bool=2, m=256, n=262144,
            p=2, rho=(-0.96,), trees=64, depth=10, q=4, noise=1e-3, objective="rff",
            hidden="hyperplane_pair"),
    4: dict(name="three-objective-ehvi", d_cont=5, d_int=5, int_levels=64, d_bool=2, m=512,
            n=1048576, p=3, rho=(-0.65, 0.1, -0.45), trees=128, depth=12, q=8, noise=1e-3,
            objective="rff", hidden="hyperplane_pair"),
    5: dict(name="kriging-believer", d_cont=5, d_int=5, int_levels=64, d_bool=2, m=512,
            n=1048576, p=2, rho=(-0.93,), trees=128, depth=12, q=8, noise=1e-3, objective="rff",
            hidden="hyperplane_pair", believer=True),
}

RFF_FEATURES = 256
RFF_LENGTHSCALE = 0.5
HIDDEN_VOLUME = 0.30
DELTA0 = 0.5
XI = 1e-4


def _streams(cfg_id):
    ss = np.random.SeedSequence([MASTER_SEED, int(cfg_id)])
    names = ["obs", "pool", "objective", "noise", "hyper", "hidden", "forest", "spare"]
    return {k: np.random.default_rng(s) for k, s in zip(names, ss.spawn(8))}


def dims(c):
    return c["d_cont"] + c["d_int"] + c["d_bool"]


def snap(U, c):
    """Round the integer and boolean dimensions of U (float64, in [0,1]) to their grids."""
    X = np.array(U, dtype=np.float64, copy=True)
    a, b = c["d_cont"], c["d_cont"] + c["d_int"]
    L = c["int_levels"] - 1
    X[:, a:b] = np.rint(X[:, a:b] * L) / L
    X[:, b:] = (X[:, b:] >= 0.5).astype(np.float64)
    return X


def _draw(rng, count, c):
    return snap(rng.random((count, dims(c))), c)


class _Objectives:
    """Seeded smooth functions on [0,1]^d returning (n, p) values."""

    def __init__(self, c, rng):
        self.c = c
        d, p = dims(c), c["p"]
        if c["objective"] == "sines":
            self.w = rng.random(d)
        else:
            D = RFF_FEATURES
            self.omega = rng.standard_normal((d, D)) / RFF_LENGTHSCALE
            self.phase = rng.random(D) * 2.0 * np.pi
            R = np.eye(p)
            rho = c.get("rho", ())
            pairs = [(0, 1), (0, 2), (1, 2)]
            for (i, j), r in zip(pairs, rho):
                R[i, j] = R[j, i] = r
            Z = rng.standard_normal((D, p))
            evals, evecs = np.linalg.eigh(R)
            R_half = evecs @ np.diag(np.sqrt(np.clip(evals, 1e-12, None))) @ evecs.T
            self.weights = Z @ R_half

    def __call__(self, X):
        if self.c["objective"] == "sines":
            return (np.sin(6.0 * X) @ self.w)[:, None]
        feats = np.sqrt(2.0 / RFF_FEATURES) * np.cos(X @ self.omega + self.phase)
        return feats @ self.weights


class _Hidden:
    """Seeded hidden-constraint region; feasible(X) -> bool array."""

    def __init__(self, c, rng):
        self.c = c
        if c["hidden"] == "halfplane":
            return
        d = dims(c)
        self.a1 = rng.standard_normal(d)
        self.a2 = rng.standard_normal(d)
        U = _draw(rng, 1_000_000, c)
        s1, s2 = U @ self.a1, U @ self.a2
        self.b2 = float(np.median(s2))
        hi2 = s2 > self.b2
        lo, hi = float(s1.min()), float(s1.max())
        for _ in range(60):
            mid = 0.5 * (lo + hi)
            vol = np.mean((s1 > mid) & hi2)
            if vol > HIDDEN_VOLUME:
                lo = mid
            else:
                hi = mid
        self.b1 = 0.5 * (lo + hi)
        self.volume = float(np.mean((s1 > self.b1) & hi2))

    def __call__(self, X):
        if self.c["hidden"] == "halfplane":
            return X[:, 0] + X[:, 3] < 1.2
        return ~((X @ self.a1 > self.b1) & (X @ self.a2 > self.b2))


def export_forest(model):
    """Flatten a fitted sklearn forest into the node arrays the scorer reads."""
    feat, thr, left, right, leaf, off = [], [], [], [], [], [0]
    for est in model.estimators_:
        t = est.tree_
        t64 = t.threshold.astype(np.float64)
        t32 = t64.astype(np.float32)
        up = t32.astype(np.float64) > t64
        t32[up] = np.nextafter(t32[up], np.float32(-np.inf))
        is_leaf = t.children_left < 0
        feat.append(np.where(is_leaf, 0, t.feature).astype(np.int32))
        thr.append(np.where(is_leaf, np.float32(0), t32).astype(np.float32))
        left.append(t.children_left.astype(np.int32))
        right.append(t.children_right.astype(np.int32))
        leaf.append(np.where(is_leaf, np.rint(t.value[:, 0, 0] * 65536.0), 0).astype(np.int32))
        off.append(off[-1] + t.node_count)
    return dict(feature=np.concatenate(feat), threshold=np.concatenate(thr),
                left=np.concatenate(left), right=np.concatenate(right),
                leaf_q16=np.concatenate(leaf), tree_offset=np.array(off, dtype=np.int64))


def levels(c):
    """Per dimension: 0 continuous, 1 boolean, L >= 2 an integer grid of L levels."""
    return [0] * c["d_cont"] + [c["int_levels"]] * c["d_int"] + [1] * c["d_bool"]


def sobol_table(d):
    """Primitive polynomials and initial direction numbers of the first d
    Sobol dimensions: the Joe-Kuo table (new-joe-kuo-6.21201) as scipy ships
    it, read with numpy's loader (no pickles).  An input of the method, like a
    seed: both the generator and its check receive it from here."""
    import glob
    import os
    import scipy
    f = glob.glob(os.path.join(os.path.dirname(scipy.__file__), "stats", "_sobol_direction_numbers.npz"))[0]
    z = np.load(f, allow_pickle=False)
    return z["poly"][:d].astype(np.int64), z["vinit"][:d].astype(np.int64)


# A vLLM-like space of nine knobs (the paper's Table 1) with the engine's
# known constraints (the paper's appendix), on 4 GPUs and a model whose
# maximum length is 4096 tokens.  Knob k takes x_k in [0, 1]; an integer knob
# with range [lo, hi] is the grid of L = hi - lo + 1 levels, value
# lo + (hi - lo) x; the block-size enumeration {8, 16, 32} is a 3-level grid
# over its indices; booleans are 0 / 1.
VLLM_KNOBS = [  # name, kind, lo, hi
    ("tensor-parallel", "int", 1, 4),
    ("max-num-seqs", "int", 64, 8192),
    ("max-num-batched-tokens", "int", 64, 8192),
    ("block-size", "enum", (8, 16, 32), None),
    ("scheduler-delay-factor", "float", 0.0, 2.0),
    ("enable-chunked-prefill", "bool", None, None),
    ("enable-prefix-caching", "bool", None, None),
    ("disable-custom-all-reduce", "bool", None, None),
    ("use-v2-block-manager", "bool", None, None),
]
VLLM_MAX_MODEL_LEN = 4096


def vllm_space():
    """levels, and the known constraints as rows A x <= b over the normalised
    knobs.  Integer inequalities get half a grid step of slack so that the
    float32 rounding of the grid points cannot flip a boundary case:

    * max-num-batched-tokens >= max-num-seqs:  x_seqs - x_tokens <= 0.5 / 8128
    * not (chunked prefill and prefix caching):  x_chunk + x_prefix <= 1
    * no chunked prefill => max-num-batched-tokens >= max model length:
      (4096 - 64 - 0.5) / 8128 - x_tokens - 2 x_chunk <= 0  (big-M, M = 2)
    """
    fixed = {"enum": 3, "float": 0, "bool": 1}
    levels = [hi - lo + 1 if kind == "int" else fixed[kind] for _, kind, lo, hi in VLLM_KNOBS]
    d = len(VLLM_KNOBS)
    A = np.zeros((3, d))
    b = np.zeros(3)
    span = 8192 - 64
    A[0, 1], A[0, 2], b[0] = 1.0, -1.0, 0.5 / span
    A[1, 5], A[1, 6], b[1] = 1.0, 1.0, 1.0
    A[2, 2], A[2, 5], b[2] = -1.0, -2.0, -(VLLM_MAX_MODEL_LEN - 64 - 0.5) / span
    return dict(levels=levels, A=A, b=b, d=d)


def space_constraints(c):
    """Known constraints of the same three shapes as the engine rules, on the
    synthetic spaces: the first integer knob at most the second (half a grid
    step of slack), not both booleans, and the third integer knob in the upper
    half unless the first boolean is set (big-M, M = 2)."""
    d = dims(c)
    i0 = c["d_cont"]
    b0 = c["d_cont"] + c["d_int"]
    A = np.zeros((3, d))
    b = np.zeros(3)
    A[0, i0], A[0, i0 + 1], b[0] = 1.0, -1.0, 0.5 / (c["int_levels"] - 1)
    A[1, b0], A[1, b0 + 1], b[1] = 1.0, 1.0, 1.0
    A[2, i0 + 2], A[2, b0], b[2] = -1.0, -2.0, -0.5
    return A, b


def vllm_decode(X):
    """Engine values of normalised configurations (float64 in, list of dicts' columns out)."""
    X = np.asarray(X, dtype=np.float64)
    cols = {}
    for k, (name, kind, lo, hi) in enumerate(VLLM_KNOBS):
        x = X[:, k]
        if kind == "int":
            cols[name] = lo + np.rint(x * (hi - lo)).astype(np.int64)
        elif kind == "enum":
            cols[name] = np.asarray(lo)[np.rint(x * (len(lo) - 1)).astype(np.int64)]
        elif kind == "float":
            cols[name] = lo + (hi - lo) * x
        else:
            cols[name] = x >= 0.5
    return cols


def make_pool(cfg_id, n=None):
    """The candidate pool alone: (n, d) float32, grid-snapped."""
    c = CONFIGS[cfg_id]
    rng = _streams(cfg_id)["pool"]
    n = c["n"] if n is None else int(n)
    return _draw(rng, n, c).astype(np.float32)


def make_workload(cfg_id, n=None, m=None, with_forest=True, kernel="matern52", warp=False):
    """Every input of one scoring pass for workload ``cfg_id``.

    ``n`` / ``m`` override the pool size / number of feasible observations
    (smaller test cases with the same recipe).  ``kernel`` names the
    covariance ("matern52" or "matern32"); ``warp`` adds per-objective,
    per-dimension input-warping parameters (a, b), log-normal around 1
    (sd 0.5 in the log), drawn from the spare stream."""
    from sklearn.ensemble import RandomForestRegressor

    c = dict(CONFIGS[cfg_id])
    if m is not None:
        c["m"] = int(m)
    rs = _streams(cfg_id)
    d, p = dims(c), c["p"]
    hidden = _Hidden(c, rs["hidden"])
    objective = _Objectives(c, rs["objective"])

    draws, labels = [], []
    feas_x = []
    while len(feas_x) < c["m"]:
        x = _draw(rs["obs"], 1, c)
        ok = bool(hidden(x)[0])
        draws.append(x[0])
        labels.append(1.0 if ok else 0.0)
        if ok:
            feas_x.append(x[0])
    X = np.array(feas_x)
    Xall = np.array(draws)
    yall = np.array(labels)
    noise_sd = np.sqrt(c["noise"]) if c["objective"] == "rff" else 0.01
    Yraw = objective(X) + noise_sd * rs["noise"].standard_normal((len(X), p))
    Y = (Yraw - Yraw.mean(axis=0)) / Yraw.std(axis=0)

    hyp = rs["hyper"]
    lengthscale = [hyp.uniform(0.1, 1.0, size=d) for _ in range(p)]

    w = dict(cfg=cfg_id, config=c, d=d, m=len(X), p=p, X=X, Y=Y, X_draws=Xall,
             feasible_draws=yall, lengthscale=lengthscale,
             signal_var=[1.0] * p, noise_var=[c["noise"]] * p, prior_mean=[0.0] * p,
             delta=DELTA0, xi=XI, q=c["q"], best_y=float(Y[:, 0].min()),
             hidden=hidden)
    if p > 1:
        mx, mn = Y.max(axis=0), Y.min(axis=0)
        w["ref"] = mx + 0.1 * (mx - mn)
    w["kernel"] = kernel
    if warp:
        sp = rs["spare"]
        w["warp"] = ([np.exp(0.5 * sp.standard_normal(d)) for _ in range(p)],
                     [np.exp(0.5 * sp.standard_normal(d)) for _ in range(p)])
    w["Xc"] = make_pool(cfg_id, n)
    if with_forest:
        seed = int(rs["forest"].integers(0, 2**31 - 1))
        model = RandomForestRegressor(n_estimators=c["trees"], max_depth=c["depth"],
                                      random_state=seed)
        model.fit(Xall, yall)
        w["forest"] = export_forest(model)
        w["forest_model"] = model
    return w
