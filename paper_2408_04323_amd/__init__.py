"""MI355X-native candidate scoring for SCOOT's suggestion step (arXiv 2408.04323).

A thin Python binding over the C ABI of ``libscoot.so`` (``include/scoot.h``):
arguments are marshalled here, every step of the scoring path runs in the
library's HIP kernels.  Device arrays are torch tensors on the current HIP
device; torch provides only memory and the stream.  Names follow the C calls
without the ``scoot_`` prefix.
"""
import ctypes as C

import numpy as np

from ._native import ScootError, check, lib  # noqa: F401

F32, F64 = 0, 1
_DT = {"f32": F32, "float32": F32, "f64": F64, "float64": F64}
MATERN52, MATERN32 = 0, 1
_KERNEL = {"matern52": MATERN52, "matern32": MATERN32}


def _kernel(kernel):
    return kernel if isinstance(kernel, int) else _KERNEL[kernel]


def _warp(warp_a, warp_b, d):
    if (warp_a is None) != (warp_b is None):
        raise ValueError("warp_a and warp_b go together")
    if warp_a is None:
        return None, None, None, None
    a, pa = _host(np.asarray(warp_a, dtype=np.float64).reshape(d), np.float64)
    b, pb = _host(np.asarray(warp_b, dtype=np.float64).reshape(d), np.float64)
    return a, b, pa, pb


def _dt(dtype):
    if isinstance(dtype, int):
        return dtype
    if not isinstance(dtype, str):
        import torch
        return F64 if dtype == torch.float64 else F32
    return _DT[dtype]


def _tdtype(dt):
    import torch
    return torch.float32 if dt == F32 else torch.float64


def _stream(stream):
    if stream is not None:
        return C.c_void_p(int(stream))
    import torch
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dptr(t):
    return C.c_void_p(0 if t is None else t.data_ptr())


def _host(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(C.POINTER(np.ctypeslib.as_ctypes_type(dtype)))


def _require_device(t, name, dtype=None, numel=None):
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} must have {numel} elements")


def abi_version():
    return lib().scoot_abi_version()


# --------------------------------------------------------------------------- fit
def gp_factor_host(X, y, lengthscale, signal_var, noise_var, prior_mean=0.0, kernel="matern52", warp_a=None,
                   warp_b=None):
    """Host fit arithmetic: returns (L, alpha) as float64 arrays."""
    X, pX = _host(X, np.float64)
    y, py = _host(y, np.float64)
    ls, pl = _host(lengthscale, np.float64)
    m, d = X.shape
    a, b, pa, pb = _warp(warp_a, warp_b, d)
    L = np.zeros((m, m))
    alpha = np.zeros(m)
    check(lib().scoot_gp_factor_host_ex(pX, py, m, d, _kernel(kernel), pl, pa, pb, signal_var, noise_var, prior_mean,
                                        L.ctypes.data_as(C.POINTER(C.c_double)),
                                        alpha.ctypes.data_as(C.POINTER(C.c_double))), "gp_factor_host")
    return L, alpha


class GP:
    """Device-resident GP state of one objective (a scoot_gp handle)."""

    def __init__(self, handle, m, d, dtype):
        self._h = C.c_void_p(handle)
        self.m, self.d, self.dtype = m, d, dtype

    @property
    def handle(self):
        return self._h

    def close(self):
        if self._h and self._h.value:
            lib().scoot_gp_destroy(self._h)
            self._h = C.c_void_p(0)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def gp_fit(X, y, lengthscale, signal_var, noise_var, prior_mean=0.0, dtype="f32", stream=None, kernel="matern52",
           warp_a=None, warp_b=None):
    """Fit on the host, GP state on the device.  kernel: "matern52" or
    "matern32" (the paper's); warp_a / warp_b: Kumaraswamy input warping."""
    X, pX = _host(X, np.float64)
    y, py = _host(y, np.float64)
    ls, pl = _host(lengthscale, np.float64)
    m, d = X.shape
    a, b, pa, pb = _warp(warp_a, warp_b, d)
    h = C.c_void_p(0)
    dt = _dt(dtype)
    check(lib().scoot_gp_fit_ex(pX, py, m, d, _kernel(kernel), pl, pa, pb, signal_var, noise_var, prior_mean, dt,
                                _stream(stream), C.byref(h)), "gp_fit")
    return GP(h.value, m, d, dt)


def gp_fit_device(X, y, lengthscale, signal_var, noise_var, prior_mean=0.0, dtype="f32", stream=None,
                  kernel="matern52", warp_a=None, warp_b=None):
    """gp_fit with the factorization, L^-1 and alpha on the current device
    (noise_var > 0)."""
    X, pX = _host(X, np.float64)
    y, py = _host(y, np.float64)
    ls, pl = _host(lengthscale, np.float64)
    m, d = X.shape
    a, b, pa, pb = _warp(warp_a, warp_b, d)
    h = C.c_void_p(0)
    dt = _dt(dtype)
    check(lib().scoot_gp_fit_device(pX, py, m, d, _kernel(kernel), pl, pa, pb, signal_var, noise_var, prior_mean,
                                    dt, _stream(stream), C.byref(h)), "gp_fit_device")
    return GP(h.value, m, d, dt)


# ---------------------------------------------------- maximum-likelihood fit
def gp_nll(X, y, theta, kernel="matern52", warp_a=None, warp_b=None, prior_mean=0.0):
    """(nll, grad) at theta = (log l_1..d, log s2, log tau2)."""
    X, pX = _host(X, np.float64)
    y, py = _host(y, np.float64)
    m, d = X.shape
    a, b, pa, pb = _warp(warp_a, warp_b, d)
    th, pt = _host(theta, np.float64)
    nll = C.c_double(0.0)
    grad = np.zeros(d + 2)
    check(lib().scoot_gp_nll(pX, py, m, d, _kernel(kernel), pa, pb, prior_mean, pt, C.byref(nll),
                             grad.ctypes.data_as(C.POINTER(C.c_double))), "gp_nll")
    return nll.value, grad


def gp_mle(X, y, theta0, lower, upper, kernel="matern52", warp_a=None, warp_b=None, prior_mean=0.0, max_iter=200):
    """Maximum-likelihood theta in [lower, upper] from theta0.  Returns (theta, nll, iterations)."""
    X, pX = _host(X, np.float64)
    y, py = _host(y, np.float64)
    m, d = X.shape
    a, b, pa, pb = _warp(warp_a, warp_b, d)
    th = np.array(theta0, dtype=np.float64).copy()
    lo, plo = _host(lower, np.float64)
    hi, phi = _host(upper, np.float64)
    nll = C.c_double(0.0)
    it = C.c_int(0)
    check(lib().scoot_gp_mle(pX, py, m, d, _kernel(kernel), pa, pb, prior_mean, plo, phi, max_iter,
                             th.ctypes.data_as(C.POINTER(C.c_double)), C.byref(nll), C.byref(it)), "gp_mle")
    return th, nll.value, it.value


def gp_nll_warp(X, y, theta, kernel="matern32", prior_mean=0.0):
    """(nll, grad) with the warping learned: theta = (log l_1..d, log s2,
    log tau2, log a_1..d, log b_1..d)."""
    X, pX = _host(X, np.float64)
    y, py = _host(y, np.float64)
    m, d = X.shape
    th, pt = _host(theta, np.float64)
    if th.size != 3 * d + 2:
        raise ValueError("theta must have 3d + 2 entries")
    nll = C.c_double(0.0)
    grad = np.zeros(3 * d + 2)
    check(lib().scoot_gp_nll_warp(pX, py, m, d, _kernel(kernel), prior_mean, pt, C.byref(nll),
                                  grad.ctypes.data_as(C.POINTER(C.c_double))), "gp_nll_warp")
    return nll.value, grad


def gp_mle_warp(X, y, theta0, lower, upper, kernel="matern32", prior_mean=0.0, max_iter=200):
    """Maximum-likelihood theta (3d + 2 entries, the warping included) in
    [lower, upper] from theta0.  Returns (theta, nll, iterations)."""
    X, pX = _host(X, np.float64)
    y, py = _host(y, np.float64)
    m, d = X.shape
    th = np.array(theta0, dtype=np.float64).copy()
    lo, plo = _host(lower, np.float64)
    hi, phi = _host(upper, np.float64)
    if not (th.size == lo.size == hi.size == 3 * d + 2):
        raise ValueError("theta0, lower and upper must have 3d + 2 entries")
    nll = C.c_double(0.0)
    it = C.c_int(0)
    check(lib().scoot_gp_mle_warp(pX, py, m, d, _kernel(kernel), prior_mean, plo, phi, max_iter,
                                  th.ctypes.data_as(C.POINTER(C.c_double)), C.byref(nll), C.byref(it)),
          "gp_mle_warp")
    return th, nll.value, it.value


def gp_nll_device(X, y, theta, kernel="matern52", warp_a=None, warp_b=None, prior_mean=0.0, learn_warp=False,
                  stream=None, with_grad=True):
    """gp_nll (learn_warp=False) or gp_nll_warp (learn_warp=True) evaluated on
    the current device; with_grad=False skips the gradient (returned as None)."""
    X, pX = _host(X, np.float64)
    y, py = _host(y, np.float64)
    m, d = X.shape
    a, b, pa, pb = _warp(warp_a, warp_b, d)
    th, pt = _host(theta, np.float64)
    P = 3 * d + 2 if learn_warp else d + 2
    if th.size != P:
        raise ValueError(f"theta must have {P} entries")
    nll = C.c_double(0.0)
    grad = np.zeros(P) if with_grad else None
    check(lib().scoot_gp_nll_device(pX, py, m, d, _kernel(kernel), pa, pb, prior_mean, int(bool(learn_warp)), pt,
                                    C.byref(nll), grad.ctypes.data_as(C.POINTER(C.c_double)) if with_grad else None,
                                    _stream(stream)),
          "gp_nll_device")
    return nll.value, grad


def gp_mle_device(X, y, theta0, lower, upper, kernel="matern52", warp_a=None, warp_b=None, prior_mean=0.0,
                  learn_warp=False, max_iter=200, stream=None):
    """gp_mle / gp_mle_warp with every likelihood evaluation on the current
    device.  Returns (theta, nll, iterations)."""
    X, pX = _host(X, np.float64)
    y, py = _host(y, np.float64)
    m, d = X.shape
    a, b, pa, pb = _warp(warp_a, warp_b, d)
    P = 3 * d + 2 if learn_warp else d + 2
    th = np.array(theta0, dtype=np.float64).copy()
    lo, plo = _host(lower, np.float64)
    hi, phi = _host(upper, np.float64)
    if not (th.size == lo.size == hi.size == P):
        raise ValueError(f"theta0, lower and upper must have {P} entries")
    nll = C.c_double(0.0)
    it = C.c_int(0)
    check(lib().scoot_gp_mle_device(pX, py, m, d, _kernel(kernel), pa, pb, prior_mean, int(bool(learn_warp)), plo,
                                    phi, max_iter, th.ctypes.data_as(C.POINTER(C.c_double)), C.byref(nll),
                                    C.byref(it), _stream(stream)), "gp_mle_device")
    return th, nll.value, it.value


# --------------------------------------------------------------------- posterior
def posterior(gp, Xc, mu=None, sigma=None, stream=None):
    """mu, sigma of the latent f at every row of Xc (n x d float32 device)."""
    import torch
    n = Xc.shape[0]
    _require_device(Xc, "Xc", torch.float32, n * gp.d)
    td = _tdtype(gp.dtype)
    mu = torch.empty(n, dtype=td, device=Xc.device) if mu is None else mu
    sigma = torch.empty(n, dtype=td, device=Xc.device) if sigma is None else sigma
    _require_device(mu, "mu", td, n)
    _require_device(sigma, "sigma", td, n)
    check(lib().scoot_posterior(gp.handle, _dptr(Xc), n, _dptr(mu), _dptr(sigma), _stream(stream)),
          "posterior")
    return mu, sigma


def acq_ei(mu, sigma, best_y, xi=1e-4, out=None, stream=None):
    import torch
    n = mu.numel()
    dt = _dt(mu.dtype)
    _require_device(mu, "mu")
    _require_device(sigma, "sigma", mu.dtype, n)
    out = torch.empty_like(mu) if out is None else out
    _require_device(out, "out", mu.dtype, n)
    check(lib().scoot_acq_ei(_dptr(mu), _dptr(sigma), n, dt, best_y, xi, _dptr(out), _stream(stream)),
          "acq_ei")
    return out


# -------------------------------------------------------------------------- EHVI
def ehvi_front(Y_obs, ref):
    """Host: (front (k x p) float64, number of boxes)."""
    r, pr = _host(ref, np.float64)
    Y, pY = _host(np.asarray(Y_obs, dtype=np.float64).reshape(-1, len(r)), np.float64)
    m, p = Y.shape
    front = np.zeros((max(m, 1), p))
    nf, nbx = C.c_int(0), C.c_int(0)
    check(lib().scoot_ehvi_front(pY, m, p, pr, front.ctypes.data_as(C.POINTER(C.c_double)), C.byref(nf),
                                 C.byref(nbx)), "ehvi_front")
    return front[:nf.value].copy(), nbx.value


def acq_ehvi(mus, sigmas, Y_obs, ref, out=None, stream=None):
    import torch
    p = len(mus)
    n = mus[0].numel()
    dt = _dt(mus[0].dtype)
    for t in list(mus) + list(sigmas):
        _require_device(t, "mu/sigma", mus[0].dtype, n)
    Y, pY = _host(Y_obs, np.float64)
    Y = Y.reshape(len(Y), p)
    r, pr = _host(ref, np.float64)
    out = torch.empty_like(mus[0]) if out is None else out
    _require_device(out, "out", mus[0].dtype, n)
    pm = (C.c_void_p * p)(*[t.data_ptr() for t in mus])
    ps = (C.c_void_p * p)(*[t.data_ptr() for t in sigmas])
    check(lib().scoot_acq_ehvi(pm, ps, p, n, dt, pY, Y.shape[0], pr, _dptr(out), _stream(stream)),
          "acq_ehvi")
    return out


# ------------------------------------------------------------------------ forest
class Forest:
    """Device-resident packed forest (a scoot_forest handle)."""

    def __init__(self, handle, n_trees, d):
        self._h = C.c_void_p(handle)
        self.n_trees, self.d = n_trees, d

    @property
    def handle(self):
        return self._h

    def close(self):
        if self._h and self._h.value:
            lib().scoot_forest_destroy(self._h)
            self._h = C.c_void_p(0)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def forest_create(feature, threshold, left, right, leaf_q16, tree_offset, d):
    f, pf = _host(feature, np.int32)
    t, pt = _host(threshold, np.float32)
    lf, pl = _host(left, np.int32)
    rt, pr = _host(right, np.int32)
    q, pq = _host(leaf_q16, np.int32)
    off, po = _host(tree_offset, np.int64)
    T = len(off) - 1
    h = C.c_void_p(0)
    check(lib().scoot_forest_create(pf, pt, pl, pr, pq, po, T, d, C.byref(h)), "forest_create")
    return Forest(h.value, T, d)


def forest_train(X, y, n_trees, max_depth, seed, bootstrap=True):
    """Host training; returns the flat arrays (feature, threshold, left, right, value, tree_offset)."""
    X, pX = _host(X, np.float64)
    y, py = _host(y, np.float64)
    n, d = X.shape
    cnt = C.c_int64(0)
    s = C.c_uint64(seed & (2 ** 64 - 1))
    check(lib().scoot_forest_train(pX, py, n, d, n_trees, max_depth, s, int(bool(bootstrap)), 0, None, None, None,
                                   None, None, None, C.byref(cnt)), "forest_train")
    k = cnt.value
    out = dict(feature=np.zeros(k, np.int32), threshold=np.zeros(k), left=np.zeros(k, np.int32),
               right=np.zeros(k, np.int32), value=np.zeros(k), tree_offset=np.zeros(n_trees + 1, np.int64))
    ptr = {k2: v.ctypes.data_as(C.POINTER(np.ctypeslib.as_ctypes_type(v.dtype))) for k2, v in out.items()}
    check(lib().scoot_forest_train(pX, py, n, d, n_trees, max_depth, s, int(bool(bootstrap)), k, ptr["feature"],
                                   ptr["threshold"], ptr["left"], ptr["right"], ptr["value"], ptr["tree_offset"],
                                   C.byref(cnt)), "forest_train")
    return out


def forest_train_create(X, y, n_trees, max_depth, seed, bootstrap=True):
    """Host training straight into a device forest handle."""
    X, pX = _host(X, np.float64)
    y, py = _host(y, np.float64)
    n, d = X.shape
    h = C.c_void_p(0)
    check(lib().scoot_forest_train_create(pX, py, n, d, n_trees, max_depth, C.c_uint64(seed & (2 ** 64 - 1)),
                                          int(bool(bootstrap)), C.byref(h)), "forest_train_create")
    return Forest(h.value, n_trees, d)


def vote_threshold(delta, n_trees):
    v = C.c_int64(0)
    check(lib().scoot_vote_threshold(delta, n_trees, C.byref(v)), "vote_threshold")
    return v.value


def rf_feasibility(forest, Xc, delta, votes=None, mask=None, leaf_idx=False, stream=None):
    """Returns (votes int32, mask uint8, leaf ids int32 (n, T) or None)."""
    import torch
    n = Xc.shape[0]
    _require_device(Xc, "Xc", torch.float32, n * forest.d)
    votes = torch.empty(n, dtype=torch.int32, device=Xc.device) if votes is None else votes
    mask = torch.empty(n, dtype=torch.uint8, device=Xc.device) if mask is None else mask
    leaves = torch.empty((n, forest.n_trees), dtype=torch.int32, device=Xc.device) if leaf_idx else None
    check(lib().scoot_rf_feasibility(forest.handle, _dptr(Xc), n, delta, _dptr(votes), _dptr(mask),
                                     _dptr(leaves), _stream(stream)), "rf_feasibility")
    return votes, mask, leaves


# ------------------------------------------------------------------------ top-q
def suggest_topq(score, mask, q, stream=None):
    """Returns device tensors (idx int64 (q,), score (q,), n_valid int32 (1,))."""
    import torch
    n = score.numel()
    _require_device(score, "score")
    if mask is not None:
        _require_device(mask, "mask", torch.uint8, n)
    idx = torch.empty(q, dtype=torch.int64, device=score.device)
    sc = torch.empty(q, dtype=score.dtype, device=score.device)
    nv = torch.empty(1, dtype=torch.int32, device=score.device)
    check(lib().scoot_suggest_topq(_dptr(score), _dptr(mask), n, _dt(score.dtype), q, _dptr(idx), _dptr(sc),
                                   _dptr(nv), _stream(stream)), "suggest_topq")
    return idx, sc, nv


def suggest_topq_noalloc(score, mask, q, idx, score_out=None, n_valid=None, stream=None):
    """As suggest_topq into caller-provided outputs (idx int64 (q,), score_out
    of the score's dtype (q,), n_valid int32 (1,)); the library allocates
    nothing in this call."""
    import torch
    n = score.numel()
    _require_device(score, "score")
    if mask is not None:
        _require_device(mask, "mask", torch.uint8, n)
    _require_device(idx, "idx", torch.int64, q)
    if score_out is not None:
        _require_device(score_out, "score_out", score.dtype, q)
    if n_valid is not None:
        _require_device(n_valid, "n_valid", torch.int32, 1)
    check(lib().scoot_suggest_topq_noalloc(_dptr(score), _dptr(mask), n, _dt(score.dtype), q, _dptr(idx),
                                           _dptr(score_out), _dptr(n_valid), _stream(stream)), "suggest_topq_noalloc")


# ---------------------------------------------------------------------- Delta
def delta_update(delta, c, k, any_invalid):
    dd, cc = C.c_double(delta), C.c_int(c)
    check(lib().scoot_delta_update(C.byref(dd), C.byref(cc), k, int(bool(any_invalid))), "delta_update")
    return dd.value, cc.value


# ------------------------------------------------------------------ whole pass
class PoolBuffers:
    """Device outputs of one scoring pass, allocated once and reused."""

    def __init__(self, n, p, q, dtype, device):
        import torch
        td = _tdtype(dtype)
        self.mu = torch.empty((p, n), dtype=td, device=device)
        self.sigma = torch.empty((p, n), dtype=td, device=device)
        self.acq = torch.empty(n, dtype=td, device=device)
        self.votes = torch.empty(n, dtype=torch.int32, device=device)
        self.mask = torch.empty(n, dtype=torch.uint8, device=device)
        self.idx = torch.empty(q, dtype=torch.int64, device=device)
        self.score = torch.empty(q, dtype=td, device=device)
        self.n_valid = torch.empty(1, dtype=torch.int32, device=device)


def score_pool(gps, forest, Xc, q, best_y=0.0, xi=1e-4, Y_obs=None, ref=None, delta=0.5, buffers=None,
               stream=None, known=None):
    """One whole pass: posterior per GP, EI (one GP) or EHVI, forest mask
    (ANDed with the known-constraint mask ``known`` when given), top-q."""
    import torch
    p = len(gps)
    n = Xc.shape[0]
    _require_device(Xc, "Xc", torch.float32, n * gps[0].d)
    if known is not None:
        _require_device(known, "known", torch.uint8, n)
    b = PoolBuffers(n, p, q, gps[0].dtype, Xc.device) if buffers is None else buffers
    hs = (C.c_void_p * p)(*[g.handle.value for g in gps])
    if p > 1:
        Y, pY = _host(Y_obs, np.float64)
        r, pr = _host(ref, np.float64)
        m_obs = Y.reshape(-1, p).shape[0]
    else:
        pY, pr, m_obs = None, None, 0
    check(lib().scoot_score_pool_ex(hs, p, forest.handle if forest is not None else None, _dptr(known), _dptr(Xc),
                                    n, best_y, xi, pY, m_obs, pr, delta, q, _dptr(b.mu), _dptr(b.sigma), _dptr(b.acq),
                                 _dptr(b.votes), _dptr(b.mask), _dptr(b.idx), _dptr(b.score), _dptr(b.n_valid),
                                 _stream(stream)), "score_pool")
    return b


# ------------------------------------------------------------- believer picks
def suggest_kb_workspace(gps, n, q):
    hs = (C.c_void_p * len(gps))(*[g.handle.value for g in gps])
    b = C.c_uint64(0)
    check(lib().scoot_suggest_kb_workspace(hs, len(gps), n, q, C.byref(b)), "suggest_kb_workspace")
    return b.value


def suggest_kb(gps, forest, Xc, q, Y_obs, ref, delta=0.5, workspace=None, stream=None, known=None, mu_out=None,
               sigma_out=None):
    """Sequential Kriging-believer picks among the feasible (and, with
    ``known``, admissible) candidates.  Returns (picks int64 (k,), EHVI at
    each pick (k,)).  ``mu_out``/``sigma_out`` (float32 (p, n) device, optional)
    receive the posterior the last scoring round was computed from."""
    import torch
    p = len(gps)
    n = Xc.shape[0]
    _require_device(Xc, "Xc", torch.float32, n * gps[0].d)
    if known is not None:
        _require_device(known, "known", torch.uint8, n)
    for t, name in ((mu_out, "mu_out"), (sigma_out, "sigma_out")):
        if t is not None:
            _require_device(t, name, torch.float32, p * n)
    hs = (C.c_void_p * p)(*[g.handle.value for g in gps])
    r, pr = _host(ref, np.float64)
    Y, pY = _host(np.asarray(Y_obs, dtype=np.float64).reshape(-1, p), np.float64)
    picks = np.full(q, -1, dtype=np.int64)
    acq = np.full(q, np.nan)
    k = C.c_int(0)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    check(lib().scoot_suggest_kb_ex(hs, p, forest.handle if forest is not None else None, _dptr(known), _dptr(Xc), n,
                                    pY, Y.shape[0],
                                 pr, delta, q, _dptr(workspace), ws_bytes,
                                 picks.ctypes.data_as(C.POINTER(C.c_int64)),
                                 acq.ctypes.data_as(C.POINTER(C.c_double)), C.byref(k), _dptr(mu_out),
                                 _dptr(sigma_out), _stream(stream)),
          "suggest_kb")
    return picks[:k.value], acq[:k.value]


# ------------------------------------------------------------- MACE (one GP)
def ucb_beta(t):
    """beta_t of the paper's UCB schedule for tuning iteration t >= 1."""
    b = C.c_double(0.0)
    check(lib().scoot_ucb_beta(int(t), C.byref(b)), "ucb_beta")
    return b.value


def acq_mace(mu, sigma, best_y, beta, xi=1e-4, out=None, stream=None):
    """Returns (ucb, pi, ei) device tensors; out = optional (ucb, pi, ei)."""
    import torch
    n = mu.numel()
    _require_device(mu, "mu")
    _require_device(sigma, "sigma", mu.dtype, n)
    ucb, pi, ei = (torch.empty_like(mu) for _ in range(3)) if out is None else out
    for t, name in ((ucb, "ucb"), (pi, "pi"), (ei, "ei")):
        _require_device(t, name, mu.dtype, n)
    check(lib().scoot_acq_mace(_dptr(mu), _dptr(sigma), n, _dt(mu.dtype), best_y, xi, beta, _dptr(ucb), _dptr(pi),
                               _dptr(ei), _stream(stream)), "acq_mace")
    return ucb, pi, ei


def pareto_front3(a, b, c, mask=None, front=None, stream=None):
    """Non-dominated flags (all three maximised).  Returns (front uint8 (n,), n_front int32 (1,))."""
    import torch
    n = a.numel()
    _require_device(a, "a")
    _require_device(b, "b", a.dtype, n)
    _require_device(c, "c", a.dtype, n)
    if mask is not None:
        _require_device(mask, "mask", torch.uint8, n)
    front = torch.empty(n, dtype=torch.uint8, device=a.device) if front is None else front
    _require_device(front, "front", torch.uint8, n)
    nf = torch.empty(1, dtype=torch.int32, device=a.device)
    check(lib().scoot_pareto_front3(_dptr(a), _dptr(b), _dptr(c), _dptr(mask), n, _dt(a.dtype), _dptr(front),
                                    _dptr(nf), _stream(stream)), "pareto_front3")
    return front, nf


def random_pick(flags, seed, q, stream=None):
    """Seeded random q flagged candidates.  Returns (idx int64 (q,), n_flagged int32 (1,))."""
    import torch
    n = flags.numel()
    _require_device(flags, "flags", torch.uint8)
    idx = torch.empty(q, dtype=torch.int64, device=flags.device)
    nf = torch.empty(1, dtype=torch.int32, device=flags.device)
    check(lib().scoot_random_pick(_dptr(flags), n, C.c_uint64(seed & (2 ** 64 - 1)), q, _dptr(idx), _dptr(nf),
                                  _stream(stream)), "random_pick")
    return idx, nf


class MaceBuffers:
    """Device outputs of one MACE suggestion, allocated once and reused."""

    def __init__(self, n, q, dtype, device):
        import torch
        td = _tdtype(dtype)
        self.mu, self.sigma, self.ucb, self.pi, self.ei = (torch.empty(n, dtype=td, device=device) for _ in range(5))
        self.votes = torch.empty(n, dtype=torch.int32, device=device)
        self.mask = torch.empty(n, dtype=torch.uint8, device=device)
        self.front = torch.empty(n, dtype=torch.uint8, device=device)
        self.idx = torch.empty(q, dtype=torch.int64, device=device)
        self.n_front = torch.empty(1, dtype=torch.int32, device=device)


def suggest_mace(gp, forest, Xc, q, best_y, beta, seed, xi=1e-4, delta=0.5, buffers=None, stream=None,
                 known=None):
    """Posterior, (ucb, pi, ei), forest mask (ANDed with ``known`` when
    given), their Pareto front, q drawn from it."""
    import torch
    n = Xc.shape[0]
    _require_device(Xc, "Xc", torch.float32, n * gp.d)
    if known is not None:
        _require_device(known, "known", torch.uint8, n)
    b = MaceBuffers(n, q, gp.dtype, Xc.device) if buffers is None else buffers
    check(lib().scoot_suggest_mace_ex(gp.handle, forest.handle if forest is not None else None, _dptr(known),
                                      _dptr(Xc), n, best_y, xi, beta, delta, C.c_uint64(seed & (2 ** 64 - 1)), q, _dptr(b.mu),
                                   _dptr(b.sigma), _dptr(b.ucb), _dptr(b.pi), _dptr(b.ei), _dptr(b.votes),
                                   _dptr(b.mask), _dptr(b.front), _dptr(b.idx), _dptr(b.n_front), _stream(stream)),
          "suggest_mace")
    return b


# ------------------------------------------------------- candidate generation
SOBOL_MAX_DEGREE = 18


def _sobol_inputs(poly, vinit, levels):
    poly = np.ascontiguousarray(np.asarray(poly, dtype=np.int64).ravel())
    d = poly.size
    if np.any(poly < 1) or np.any(poly >= 2 ** 32):
        raise ValueError("sobol: polynomials must be positive 32-bit integers")
    vi = np.zeros((d, SOBOL_MAX_DEGREE), dtype=np.uint32)
    v = np.asarray(vinit, dtype=np.int64).reshape(d, -1)
    k = min(v.shape[1], SOBOL_MAX_DEGREE)
    if np.any(v[:, :k] < 0) or np.any(v[:, :k] >= 2 ** 32):
        raise ValueError("sobol: initial direction numbers must be 32-bit")
    vi[:, :k] = v[:, :k]
    lv = np.ascontiguousarray(np.asarray(levels, dtype=np.int32).ravel())
    if lv.size != d:
        raise ValueError("sobol: one level count per dimension")
    return np.ascontiguousarray(poly.astype(np.uint32)), vi, lv, d


def _constraint_inputs(A, b, d):
    if A is None:
        return None, None, 0
    A = np.ascontiguousarray(np.asarray(A, dtype=np.float64).reshape(-1, d))
    b = np.ascontiguousarray(np.asarray(b, dtype=np.float64).ravel())
    if b.size != A.shape[0]:
        raise ValueError("known constraints: one bound per row")
    return A, b, A.shape[0]


def sobol_pool(poly, vinit, levels, n, skip=0, A=None, b=None, device="cuda", out=None, known=None,
               with_known=None, stream=None):
    """Sobol points skip .. skip + n - 1 on the grids ``levels`` as a float32
    (n, d) device tensor, and (when constraints A x <= b are given, or
    with_known) their admissibility mask.  Returns (Xc, known or None)."""
    import torch
    pu, vi, lv, d = _sobol_inputs(poly, vinit, levels)
    A, bb, r = _constraint_inputs(A, b, d)
    Xc = torch.empty((n, d), dtype=torch.float32, device=device) if out is None else out
    _require_device(Xc, "Xc", torch.float32, n * d)
    if with_known is None:
        with_known = r > 0 or known is not None
    if with_known and known is None:
        known = torch.empty(n, dtype=torch.uint8, device=Xc.device)
    if known is not None:
        _require_device(known, "known", torch.uint8, n)
    pA = A.ctypes.data_as(C.POINTER(C.c_double)) if r else None
    pb = bb.ctypes.data_as(C.POINTER(C.c_double)) if r else None
    check(lib().scoot_sobol_pool(pu.ctypes.data_as(C.POINTER(C.c_uint32)), vi.ctypes.data_as(C.POINTER(C.c_uint32)),
                                 d, lv.ctypes.data_as(C.POINTER(C.c_int32)), int(skip), int(n), pA, pb, r, _dptr(Xc),
                                 _dptr(known), _stream(stream)), "sobol_pool")
    return Xc, known


def known_constraints(Xc, A, b, out=None, stream=None):
    """uint8 (n,) device mask: 1 where every row of A x <= b holds."""
    import torch
    n, d = Xc.shape
    _require_device(Xc, "Xc", torch.float32, n * d)
    A, bb, r = _constraint_inputs(A, b, d)
    known = torch.empty(n, dtype=torch.uint8, device=Xc.device) if out is None else out
    _require_device(known, "known", torch.uint8, n)
    pA = A.ctypes.data_as(C.POINTER(C.c_double)) if r else None
    pb = bb.ctypes.data_as(C.POINTER(C.c_double)) if r else None
    check(lib().scoot_known_constraints(_dptr(Xc), n, d, pA, pb, r, _dptr(known), _stream(stream)),
          "known_constraints")
    return known


# ------------------------------------------------------ the suggestion step
class _Space(C.Structure):
    _fields_ = [("d", C.c_int), ("levels", C.POINTER(C.c_int32)), ("sobol_poly", C.POINTER(C.c_uint32)),
                ("sobol_vinit", C.POINTER(C.c_uint32)), ("A", C.POINTER(C.c_double)),
                ("b", C.POINTER(C.c_double)), ("r", C.c_int)]


class _SuggestOpts(C.Structure):
    _fields_ = [("k", C.c_int), ("delta", C.c_double), ("pool_size", C.c_int64), ("pool_skip", C.c_int64),
                ("kernel", C.c_int), ("dtype", C.c_int), ("warp_a", C.POINTER(C.c_double)),
                ("warp_b", C.POINTER(C.c_double)), ("theta_lower", C.POINTER(C.c_double)),
                ("theta_upper", C.POINTER(C.c_double)), ("theta_start", C.POINTER(C.c_double)),
                ("mle_max_iter", C.c_int), ("n_trees", C.c_int), ("max_depth", C.c_int),
                ("forest_seed", C.c_uint64), ("bootstrap", C.c_int), ("xi", C.c_double), ("t", C.c_int),
                ("pick_seed", C.c_uint64), ("ref", C.POINTER(C.c_double)), ("learn_warp", C.c_int),
                ("host_search", C.c_int)]


def suggest(X_obs, Y_obs, valid, space, k, delta=0.5, pool_size=262144, pool_skip=0, kernel="matern52",
            dtype="f32", warp_a=None, warp_b=None, theta_lower=None, theta_upper=None, theta_start=None,
            mle_max_iter=0, n_trees=64, max_depth=10, forest_seed=0, bootstrap=True, xi=1e-4, t=1, pick_seed=0,
            ref=None, stream=None, learn_warp=False, host_search=False):
    """One SUGGEST of Algorithm 1 (scoot_suggest).  ``space`` is a dict with
    ``levels``, ``poly``, ``vinit`` and optionally ``A``, ``b`` (known
    constraints).  X_obs (n_obs, d), Y_obs (n_obs, p) minimised, valid (n_obs,)
    host arrays; per-objective options (warps (p, d), theta bounds (p, d + 2))
    host arrays; learn_warp: the warping is learned with the other
    hyperparameters; host_search: the likelihood search evaluates on the host
    instead of the device.  Returns (x (n_out, d) float64, source (n_out,) int32,
    theta (p, d + 2), or (p, 3d + 2) with learn_warp, float64)."""
    pu, vi, lv, d = _sobol_inputs(space["poly"], space["vinit"], space["levels"])
    A, bb, r = _constraint_inputs(space.get("A"), space.get("b"), d)
    X = np.ascontiguousarray(np.asarray(X_obs, dtype=np.float64).reshape(-1, d))
    n_obs = X.shape[0]
    Y = np.asarray(Y_obs, dtype=np.float64)
    p = Y.shape[1] if Y.ndim == 2 else 1
    Y = np.ascontiguousarray(Y.reshape(n_obs, p))
    ok = np.ascontiguousarray(np.asarray(valid).reshape(n_obs) != 0, dtype=np.uint8)
    keep = []  # host buffers referenced by the structures during the call

    def arr(a, shape):
        if a is None:
            return None
        h, ptr = _host(np.asarray(a, dtype=np.float64).reshape(shape), np.float64)
        keep.append(h)
        return ptr

    sp = _Space(d, lv.ctypes.data_as(C.POINTER(C.c_int32)), pu.ctypes.data_as(C.POINTER(C.c_uint32)),
                vi.ctypes.data_as(C.POINTER(C.c_uint32)),
                A.ctypes.data_as(C.POINTER(C.c_double)) if r else None,
                bb.ctypes.data_as(C.POINTER(C.c_double)) if r else None, r)
    if (warp_a is None) != (warp_b is None):
        raise ValueError("warp_a and warp_b go together")
    op = _SuggestOpts(int(k), float(delta), int(pool_size), int(pool_skip), _kernel(kernel), _dt(dtype),
                      arr(warp_a, (p, d)), arr(warp_b, (p, d)), arr(theta_lower, (p, d + 2)),
                      arr(theta_upper, (p, d + 2)), arr(theta_start, (p, d + 2)), int(mle_max_iter), int(n_trees),
                      int(max_depth), int(forest_seed), int(bool(bootstrap)), float(xi), int(t), int(pick_seed),
                      arr(ref, (p,)), int(bool(learn_warp)), int(bool(host_search)))
    x = np.zeros((k, d), dtype=np.float64)
    src = np.zeros(k, dtype=np.int32)
    theta = np.zeros((p, 3 * d + 2 if learn_warp else d + 2), dtype=np.float64)
    n_out = C.c_int(0)
    check(lib().scoot_suggest(X.ctypes.data_as(C.POINTER(C.c_double)), Y.ctypes.data_as(C.POINTER(C.c_double)),
                              ok.ctypes.data_as(C.POINTER(C.c_uint8)), n_obs, p, C.byref(sp), C.byref(op),
                              x.ctypes.data_as(C.POINTER(C.c_double)), src.ctypes.data_as(C.POINTER(C.c_int32)),
                              theta.ctypes.data_as(C.POINTER(C.c_double)), C.byref(n_out), _stream(stream)),
          "suggest")
    return x[:n_out.value], src[:n_out.value], theta
