// Maximum-likelihood GP hyperparameters on the host, fp64 (Sec. 4.3: the noise
// level tau^2 is learned by maximum likelihood; the signal variance and the
// lengthscales are learned with it).
//
// theta = (log l_1 .. log l_d, log s2, log tau2).  With K = k_theta(X, X) +
// tau2 I on the (optionally warped) inputs and r = y - c:
//   NLL = 1/2 r^T K^-1 r + 1/2 log det K + m/2 log(2 pi)
//   dNLL/dtheta_j = -1/2 sum_ik W_ik (dK/dtheta_j)_ik,  W = alpha alpha^T - K^-1
// dK/dlog s2 = K - tau2 I, dK/dlog tau2 = tau2 I, and per lengthscale
// (D_k = (x_k - x'_k) / l_k, r the scaled distance):
//   Matern-5/2: 5/3 s2 (1 + sqrt5 r) exp(-sqrt5 r) D_k^2
//   Matern-3/2: 3 s2 exp(-sqrt3 r) D_k^2.
//
// With the input warping learned as well (the paper's Matern-3/2 with input
// warping after Snoek et al., whose warp parameters are fitted with the GP),
// theta gains (log a_1 .. log a_d, log b_1 .. log b_d): the inputs are warped
// by w = 1 - (1 - x^a)^b at every evaluation, and since dk/dw_ik =
// -R_ij (w_ik - w_jk) / l_k^2 with R the radial factor above,
//   dK_ij/dlog a_k = -R_ij (w_ik - w_jk) (g_ik - g_jk) / l_k^2,
// g_ik = dw_ik/dlog a_k = a b (1 - x^a)^(b-1) x^a ln x (likewise for log b_k
// with dw/dlog b = -b (1 - x^a)^b ln(1 - x^a)), both 0 at x = 0 and 1.
//
// The search runs unconstrained L-BFGS (10 pairs, backtracking line search
// with the Armijo condition) in z with theta = lo + (hi - lo) sigmoid(z), so
// every iterate stays inside the box [lo, hi]; a parameter with lo == hi is
// held fixed.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <deque>
#include <vector>

#include "host_blas.h"
#include "internal.h"

namespace scoot {

namespace {
constexpr double kSqrt5m = 2.23606797749978969641;
constexpr double kSqrt3m = 1.73205080756887729353;
constexpr double kLog2Pi = 1.83787706640934548356;

struct MleData {
  int m, d;
  scoot_kernel kernel;
  bool learn_warp = false;  // theta carries log a, log b; Xw is recomputed per evaluation
  std::vector<double> X;   // m x d inputs as given (learn_warp)
  mutable std::vector<double> Xw;  // m x d warped inputs
  mutable std::vector<double> Ga, Gb;  // m x d: dw/dlog a, dw/dlog b (learn_warp)
  std::vector<double> r;   // y - c
  // Work matrices of nll_eval (m x m), allocated on the first evaluation and
  // reused: fresh allocations of this size are page-faulted in on every
  // evaluation, by all threads at once.  The entries an evaluation does not
  // write keep their initial zeros.
  mutable std::vector<double> L, Kf, Rad, Lt;
};

std::vector<double>& work(std::vector<double>& v, size_t n) {
  if (v.size() != n) v.assign(n, 0.0);
  return v;
}

constexpr int kChunks = 32;  // work split of every parallel step (independent of the thread count)

// The warp of x and its derivatives in log a and log b (0 at x = 0 and 1),
// written without cancellation: ln x from log1p(x - 1) above 1/2, 1 - x^a =
// -expm1(a ln x).
void warp_with_derivatives(double x, double a, double b, double* w, double* ga, double* gb) {
  x = x < 0.0 ? 0.0 : (x > 1.0 ? 1.0 : x);
  *w = kumaraswamy(x, a, b);
  if (x <= 0.0 || x >= 1.0) {
    *ga = *gb = 0.0;
    return;
  }
  const double lx = x > 0.5 ? std::log1p(x - 1.0) : std::log(x);
  const double u = std::exp(a * lx);
  const double l1u = std::log(-std::expm1(a * lx));  // ln(1 - x^a)
  *ga = a * b * std::exp((b - 1.0) * l1u) * u * lx;
  *gb = -b * std::exp(b * l1u) * l1u;
}

// NLL and gradient at theta; false when K is not positive definite.
bool nll_eval(const MleData& D, const double* theta, double* nll, double* grad) {
  const int m = D.m, d = D.d;
  double inv_ls[SCOOT_MAX_DIM];
  for (int k = 0; k < d; ++k) inv_ls[k] = std::exp(-theta[k]);
  const double s2 = std::exp(theta[d]), tau2 = std::exp(theta[d + 1]);
  const bool m52 = D.kernel == SCOOT_MATERN52;
  const double root = m52 ? kSqrt5m : kSqrt3m;
  if (D.learn_warp) {
    work(D.Xw, (size_t)m * d);
    work(D.Ga, (size_t)m * d);
    work(D.Gb, (size_t)m * d);
    for (int k = 0; k < d; ++k) {
      const double a = std::exp(theta[d + 2 + k]), b = std::exp(theta[2 * d + 2 + k]);
      for (int i = 0; i < m; ++i) {
        const size_t at = (size_t)i * d + k;
        warp_with_derivatives(D.X[at], a, b, &D.Xw[at], &D.Ga[at], &D.Gb[at]);
      }
    }
  }
  const double* X = D.Xw.data();
  const int P = D.learn_warp ? 3 * d + 2 : d + 2;

  // K (lower triangle), rows in parallel, then its Cholesky factor.  The
  // gradient reuses K - tau2 I (= dK/dlog s2) and the radial factor of
  // dK/dlog l_k, kept from here (lower triangles).
  std::vector<double>& L = work(D.L, (size_t)m * m);
  double* Kf = grad ? work(D.Kf, (size_t)m * m).data() : nullptr;
  double* Rad = grad ? work(D.Rad, (size_t)m * m).data() : nullptr;
  parallel_chunks(kChunks, [&](int c) {
    for (int i = c; i < m; i += kChunks)
      for (int j = 0; j <= i; ++j) {
        double r2 = 0.0;
        for (int k = 0; k < d; ++k) {
          const double t = (X[(size_t)i * d + k] - X[(size_t)j * d + k]) * inv_ls[k];
          r2 += t * t;
        }
        const double t = root * std::sqrt(r2);
        const double e = std::exp(-t);
        const double kv = m52 ? s2 * (1.0 + t + t * t / 3.0) * e : s2 * (1.0 + t) * e;
        L[(size_t)i * m + j] = kv + (i == j ? tau2 : 0.0);
        if (grad) {
          Kf[(size_t)i * m + j] = kv;
          Rad[(size_t)i * m + j] = m52 ? 5.0 / 3.0 * s2 * (1.0 + t) * e : 3.0 * s2 * e;
        }
      }
  });
  if (!cholesky_lower(L.data(), m)) return false;

  // alpha = K^-1 r and log det K: forward substitution by rows, back
  // substitution by columns of L^T (rows of L, contiguous).
  std::vector<double> z(m), alpha(m);
  double logdet = 0.0;
  for (int i = 0; i < m; ++i) {
    const double* Li = L.data() + (size_t)i * m;
    z[i] = (D.r[i] - dot2(Li, z.data(), i)) / Li[i];
    logdet += 2.0 * std::log(Li[i]);
  }
  alpha = z;
  for (int i = m - 1; i >= 0; --i) {
    const double* Li = L.data() + (size_t)i * m;
    alpha[i] /= Li[i];
    const double ai = alpha[i];
    for (int k = 0; k < i; ++k) alpha[k] -= Li[k] * ai;
  }
  double quad = 0.0;
  for (int i = 0; i < m; ++i) quad += D.r[i] * alpha[i];
  *nll = 0.5 * quad + 0.5 * logdet + 0.5 * m * kLog2Pi;
  if (!grad) return true;

  // K^-1 = L^-T L^-1.  Column j of L^-1 is stored as row j of Lt (zero before
  // index j), so K^-1[i][j] = sum_{k >= i} Lt[i][k] Lt[j][k] for j <= i; the
  // entries come in tiles of 4 rows x 2 columns summed from the tile's first
  // row i0 (the terms below row i are zeros).
  std::vector<double>& Lt = work(D.Lt, (size_t)m * m);
  lower_inverse(L.data(), m, Lt.data(), true);

  // Gradient: tiles by groups of four rows, partial sums per chunk, added in
  // chunk order.
  std::vector<double> part((size_t)kChunks * P, 0.0);
  const int groups = (m + 3) / 4;
  const double* Ga = D.learn_warp ? D.Ga.data() : nullptr;
  const double* Gb = D.learn_warp ? D.Gb.data() : nullptr;
  parallel_chunks(kChunks, [&](int c) {
    double* g = part.data() + (size_t)c * P;
    for (int gi = c; gi < groups; gi += kChunks) {
      const int i0 = 4 * gi;
      const double* a[4];
      for (int r = 0; r < 4; ++r) a[r] = Lt.data() + (size_t)std::min(i0 + r, m - 1) * m + i0;
      for (int j0 = 0; j0 <= i0 + 3 && j0 < m; j0 += 2) {
        const double* b[2] = {Lt.data() + (size_t)j0 * m + i0, Lt.data() + (size_t)std::min(j0 + 1, m - 1) * m + i0};
        double kinv[4][2];
        dots_tile<4, 2>(a, b, m - i0, kinv);
        for (int r = 0; r < 4; ++r)
          for (int q = 0; q < 2; ++q) {
            const int i = i0 + r, j = j0 + q;
            if (i >= m || j > i) continue;
            const double Wij = alpha[i] * alpha[j] - kinv[r][q];
            const double w = 0.5 * (i == j ? 1.0 : 2.0) * Wij;  // W and dK are symmetric
            const double wr = w * Rad[(size_t)i * m + j];
            for (int k = 0; k < d; ++k) {
              const double t = (X[(size_t)i * d + k] - X[(size_t)j * d + k]) * inv_ls[k];
              g[k] -= wr * (t * t);
              if (Ga) {
                const double wt = wr * t * inv_ls[k];
                g[d + 2 + k] += wt * (Ga[(size_t)i * d + k] - Ga[(size_t)j * d + k]);
                g[2 * d + 2 + k] += wt * (Gb[(size_t)i * d + k] - Gb[(size_t)j * d + k]);
              }
            }
            g[d] -= w * Kf[(size_t)i * m + j];
            if (i == j) g[d + 1] -= w * tau2;
          }
      }
    }
  });
  for (int k = 0; k < P; ++k) {
    double s = 0.0;
    for (int c = 0; c < kChunks; ++c) s += part[(size_t)c * P + k];
    grad[k] = s;
  }
  return true;
}

int prepare(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
            const double* warp_b, double c, MleData& D, bool learn_warp = false) {
  if (!X || !y) return fail(SCOOT_ERR_INVALID_ARG, "gp mle: null pointer");
  if (m < 1 || d < 1) return fail(SCOOT_ERR_INVALID_ARG, "gp mle: m and d must be >= 1");
  if (d > SCOOT_MAX_DIM) return fail(SCOOT_ERR_UNSUPPORTED, "gp mle: d exceeds SCOOT_MAX_DIM");
  if (m > SCOOT_MAX_OBS) return fail(SCOOT_ERR_UNSUPPORTED, "gp mle: m exceeds SCOOT_MAX_OBS");
  if (kernel != SCOOT_MATERN52 && kernel != SCOOT_MATERN32) return fail(SCOOT_ERR_INVALID_ARG, "gp mle: bad kernel");
  if ((warp_a == nullptr) != (warp_b == nullptr))
    return fail(SCOOT_ERR_INVALID_ARG, "gp mle: warp_a and warp_b go together");
  for (size_t i = 0; i < (size_t)m * d; ++i)
    if (!std::isfinite(X[i])) return fail(SCOOT_ERR_INVALID_ARG, "gp mle: non-finite observation");
  for (int i = 0; i < m; ++i)
    if (!std::isfinite(y[i])) return fail(SCOOT_ERR_INVALID_ARG, "gp mle: non-finite observation");
  if (!std::isfinite(c)) return fail(SCOOT_ERR_INVALID_ARG, "gp mle: non-finite prior mean");
  if (warp_a)
    for (int k = 0; k < d; ++k)
      if (!(warp_a[k] > 0) || !(warp_b[k] > 0) || !std::isfinite(warp_a[k]) || !std::isfinite(warp_b[k]))
        return fail(SCOOT_ERR_INVALID_ARG, "gp mle: warping parameters must be finite and > 0");
  D.m = m;
  D.d = d;
  D.kernel = kernel;
  D.learn_warp = learn_warp;
  if (learn_warp) D.X.assign(X, X + (size_t)m * d);
  D.Xw.assign(X, X + (size_t)m * d);
  if (warp_a)
    for (int i = 0; i < m; ++i)
      for (int k = 0; k < d; ++k) D.Xw[(size_t)i * d + k] = kumaraswamy(X[(size_t)i * d + k], warp_a[k], warp_b[k]);
  D.r.resize(m);
  for (int i = 0; i < m; ++i) D.r[i] = y[i] - c;
  return SCOOT_OK;
}

double sigmoid(double z) { return z >= 0 ? 1.0 / (1.0 + std::exp(-z)) : std::exp(z) / (1.0 + std::exp(z)); }
}  // namespace

int mle_nll(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
            const double* warp_b, double c, const double* theta, double* nll, double* grad, bool learn_warp) {
  if (!theta || !nll) return fail(SCOOT_ERR_INVALID_ARG, "gp nll: null pointer");
  MleData D;
  int rc = prepare(X, y, m, d, kernel, warp_a, warp_b, c, D, learn_warp);
  if (rc != SCOOT_OK) return rc;
  for (int k = 0; k < (learn_warp ? 3 * d + 2 : d + 2); ++k)
    if (!std::isfinite(theta[k])) return fail(SCOOT_ERR_INVALID_ARG, "gp nll: non-finite theta");
  if (!nll_eval(D, theta, nll, grad)) return fail(SCOOT_ERR_NOT_PD, "gp nll: K is not positive definite");
  return SCOOT_OK;
}

int mle_inputs(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
               const double* warp_b, double c, bool learn_warp, std::vector<double>& Xuse, std::vector<double>& r) {
  MleData D;
  int rc = prepare(X, y, m, d, kernel, warp_a, warp_b, c, D, learn_warp);
  if (rc != SCOOT_OK) return rc;
  Xuse = learn_warp ? D.X : D.Xw;
  r = D.r;
  return SCOOT_OK;
}

int mle_fit(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
            const double* warp_b, double c, const double* lower, const double* upper, int max_iter, double* theta,
            double* nll_out, int* iters_out, bool learn_warp) {
  if (!lower || !upper || !theta) return fail(SCOOT_ERR_INVALID_ARG, "gp mle: null pointer");
  if (max_iter < 1) return fail(SCOOT_ERR_INVALID_ARG, "gp mle: max_iter must be >= 1");
  MleData D;
  int rc = prepare(X, y, m, d, kernel, warp_a, warp_b, c, D, learn_warp);
  if (rc != SCOOT_OK) return rc;
  const int P = learn_warp ? 3 * d + 2 : d + 2;
  return lbfgs_box([&](const double* t, double* f, double* g) { return nll_eval(D, t, f, g); }, P, lower, upper,
                   max_iter, theta, nll_out, iters_out);
}

int lbfgs_box(const NllFn& nll_fn, int P, const double* lower, const double* upper, int max_iter, double* theta,
              double* nll_out, int* iters_out) {
  if (!lower || !upper || !theta) return fail(SCOOT_ERR_INVALID_ARG, "gp mle: null pointer");
  if (max_iter < 1) return fail(SCOOT_ERR_INVALID_ARG, "gp mle: max_iter must be >= 1");
  for (int k = 0; k < P; ++k)
    if (!std::isfinite(lower[k]) || !std::isfinite(upper[k]) || lower[k] > upper[k] || !std::isfinite(theta[k]))
      return fail(SCOOT_ERR_INVALID_ARG, "gp mle: bounds must be finite with lower <= upper, theta finite");
  // free parameters and their z coordinates
  std::vector<int> fr;
  for (int k = 0; k < P; ++k)
    if (upper[k] > lower[k]) fr.push_back(k);
  const int F = (int)fr.size();
  std::vector<double> th(theta, theta + P);
  std::vector<double> z(F);
  for (int f = 0; f < F; ++f) {
    const int k = fr[f];
    double u = (std::min(std::max(th[k], lower[k]), upper[k]) - lower[k]) / (upper[k] - lower[k]);
    u = std::min(std::max(u, 1e-9), 1.0 - 1e-9);
    z[f] = std::log(u / (1.0 - u));
  }
  for (int k = 0; k < P; ++k)
    if (upper[k] == lower[k]) th[k] = lower[k];
  auto to_theta = [&](const std::vector<double>& zz, std::vector<double>& t) {
    t = th;
    for (int f = 0; f < F; ++f) t[fr[f]] = lower[fr[f]] + (upper[fr[f]] - lower[fr[f]]) * sigmoid(zz[f]);
  };
  std::vector<double> gth(P), t(P);
  auto eval = [&](const std::vector<double>& zz, double& f, std::vector<double>& gz) {
    to_theta(zz, t);
    if (!nll_fn(t.data(), &f, gth.data())) return false;
    gz.assign(F, 0.0);
    for (int q = 0; q < F; ++q) {
      const int k = fr[q];
      const double s = sigmoid(zz[q]);
      gz[q] = gth[k] * (upper[k] - lower[k]) * s * (1.0 - s);
    }
    return true;
  };

  double f;
  std::vector<double> g;
  if (!eval(z, f, g)) return fail(SCOOT_ERR_NOT_PD, "gp mle: K is not positive definite at the start");
  std::deque<std::vector<double>> S, Y;
  int it = 0;
  // A parameter pushed against a bound sits where the sigmoid is flat, so its
  // z-gradient vanishes even where the likelihood still falls inwards: after
  // the search stops, such parameters are moved 1% of their range inside and
  // the search restarts (fresh history), up to kRestarts times; the best
  // point seen is returned.
  constexpr int kRestarts = 4;
  std::vector<double> z_best = z;
  double f_best = f;
  for (int restart = 0; restart <= kRestarts; ++restart) {
    for (; it < max_iter && F > 0; ++it) {
      double gmax = 0.0;
      for (double v : g) gmax = std::max(gmax, std::fabs(v));
      if (gmax < 1e-9) break;
      // two-loop recursion: p = -H g
      std::vector<double> q = g;
      const int h = (int)S.size();
      std::vector<double> al(h), rho(h);
      for (int i = h - 1; i >= 0; --i) {
        double sy = 0, sq = 0;
        for (int k = 0; k < F; ++k) {
          sy += S[i][k] * Y[i][k];
          sq += S[i][k] * q[k];
        }
        rho[i] = 1.0 / sy;
        al[i] = rho[i] * sq;
        for (int k = 0; k < F; ++k) q[k] -= al[i] * Y[i][k];
      }
      double gamma = 1.0;
      if (h > 0) {
        double sy = 0, yy = 0;
        for (int k = 0; k < F; ++k) {
          sy += S[h - 1][k] * Y[h - 1][k];
          yy += Y[h - 1][k] * Y[h - 1][k];
        }
        gamma = sy / yy;
      }
      for (int k = 0; k < F; ++k) q[k] *= gamma;
      for (int i = 0; i < h; ++i) {
        double yq = 0;
        for (int k = 0; k < F; ++k) yq += Y[i][k] * q[k];
        const double b = rho[i] * yq;
        for (int k = 0; k < F; ++k) q[k] += S[i][k] * (al[i] - b);
      }
      std::vector<double> p(F);
      double gp = 0;
      for (int k = 0; k < F; ++k) {
        p[k] = -q[k];
        gp += p[k] * g[k];
      }
      if (!(gp < 0)) {  // not a descent direction: restart from steepest descent
        S.clear();
        Y.clear();
        gp = 0;
        for (int k = 0; k < F; ++k) {
          p[k] = -g[k];
          gp -= g[k] * g[k];
        }
      }
      // step: at most 2 in z per coordinate on the first iteration
      double step = 1.0;
      if (h == 0) {
        double pmax = 0;
        for (double v : p) pmax = std::max(pmax, std::fabs(v));
        if (pmax > 2.0) step = 2.0 / pmax;
      }
      std::vector<double> zn(F), gn;
      double fn = 0;
      bool ok = false;
      for (int ls = 0; ls < 40; ++ls, step *= 0.5) {
        for (int k = 0; k < F; ++k) zn[k] = z[k] + step * p[k];
        if (eval(zn, fn, gn) && fn <= f + 1e-4 * step * gp) {
          ok = true;
          break;
        }
      }
      if (!ok) break;  // no decrease along p: converged to rounding
      std::vector<double> s(F), yv(F);
      double sy = 0;
      for (int k = 0; k < F; ++k) {
        s[k] = zn[k] - z[k];
        yv[k] = gn[k] - g[k];
        sy += s[k] * yv[k];
      }
      if (sy > 1e-14) {
        S.push_back(s);
        Y.push_back(yv);
        if (S.size() > 10) {
          S.pop_front();
          Y.pop_front();
        }
      }
      const double df = f - fn;
      z = zn;
      f = fn;
      g = gn;
      if (df <= 1e-13 * std::max(1.0, std::fabs(f))) {
        ++it;
        break;
      }
    }
    if (f < f_best) {
      f_best = f;
      z_best = z;
    }
    if (restart == kRestarts || it >= max_iter || F == 0) break;
    // the gradient in theta at the point reached (eval leaves it in gth)
    double f_here;
    std::vector<double> g_here;
    if (!eval(z, f_here, g_here)) break;
    bool moved = false;
    for (int q = 0; q < F; ++q) {
      const double u = sigmoid(z[q]), gk = gth[fr[q]];
      if (u > 1.0 - 1e-6 && gk > 0) {
        z[q] = std::log(0.99 / 0.01);
        moved = true;
      } else if (u < 1e-6 && gk < 0) {
        z[q] = std::log(0.01 / 0.99);
        moved = true;
      }
    }
    if (!moved || !eval(z, f, g)) break;
    S.clear();
    Y.clear();
  }
  to_theta(z_best, t);
  std::memcpy(theta, t.data(), sizeof(double) * P);
  if (nll_out) *nll_out = f_best;
  if (iters_out) *iters_out = it;
  return SCOOT_OK;
}

}  // namespace scoot
