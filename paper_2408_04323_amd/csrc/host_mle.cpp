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
// The search runs unconstrained L-BFGS (10 pairs, backtracking line search
// with the Armijo condition) in z with theta = lo + (hi - lo) sigmoid(z), so
// every iterate stays inside the box [lo, hi]; a parameter with lo == hi is
// held fixed.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <deque>
#include <vector>

#include "internal.h"

namespace scoot {

namespace {
constexpr double kSqrt5m = 2.23606797749978969641;
constexpr double kSqrt3m = 1.73205080756887729353;
constexpr double kLog2Pi = 1.83787706640934548356;

struct MleData {
  int m, d;
  scoot_kernel kernel;
  std::vector<double> Xw;  // m x d warped inputs
  std::vector<double> r;   // y - c
};

constexpr int kChunks = 32;  // work split of every parallel step (independent of the thread count)

double dot(const double* a, const double* b, int n) {
  double s = 0.0;
#pragma omp simd reduction(+ : s)
  for (int k = 0; k < n; ++k) s += a[k] * b[k];
  return s;
}

// NLL and gradient at theta; false when K is not positive definite.
bool nll_eval(const MleData& D, const double* theta, double* nll, double* grad) {
  const int m = D.m, d = D.d;
  double inv_ls[SCOOT_MAX_DIM];
  for (int k = 0; k < d; ++k) inv_ls[k] = std::exp(-theta[k]);
  const double s2 = std::exp(theta[d]), tau2 = std::exp(theta[d + 1]);
  const bool m52 = D.kernel == SCOOT_MATERN52;
  const double root = m52 ? kSqrt5m : kSqrt3m;
  const double* X = D.Xw.data();

  // K (lower triangle), rows in parallel, then its Cholesky factor
  std::vector<double> L((size_t)m * m, 0.0);
  parallel_chunks(kChunks, [&](int c) {
    for (int i = c; i < m; i += kChunks)
      for (int j = 0; j <= i; ++j) {
        double r2 = 0.0;
        for (int k = 0; k < d; ++k) {
          const double t = (X[(size_t)i * d + k] - X[(size_t)j * d + k]) * inv_ls[k];
          r2 += t * t;
        }
        const double t = root * std::sqrt(r2);
        const double kv = m52 ? s2 * (1.0 + t + t * t / 3.0) * std::exp(-t) : s2 * (1.0 + t) * std::exp(-t);
        L[(size_t)i * m + j] = kv + (i == j ? tau2 : 0.0);
      }
  });
  if (!cholesky_lower(L.data(), m)) return false;

  // alpha = K^-1 r and log det K
  std::vector<double> z(m), alpha(m);
  double logdet = 0.0;
  for (int i = 0; i < m; ++i) {
    const double* Li = L.data() + (size_t)i * m;
    z[i] = (D.r[i] - dot(Li, z.data(), i)) / Li[i];
    logdet += 2.0 * std::log(Li[i]);
  }
  for (int i = m - 1; i >= 0; --i) {
    double s = z[i];
    for (int k = i + 1; k < m; ++k) s -= L[(size_t)k * m + i] * alpha[k];
    alpha[i] = s / L[(size_t)i * m + i];
  }
  double quad = 0.0;
  for (int i = 0; i < m; ++i) quad += D.r[i] * alpha[i];
  *nll = 0.5 * quad + 0.5 * logdet + 0.5 * m * kLog2Pi;
  if (!grad) return true;

  // K^-1 = L^-T L^-1.  Column j of L^-1 (forward substitution, columns
  // independent) is stored as row j of Lt, so that
  // K^-1[i][j] = sum_{k >= max(i, j)} Lt[i][k] Lt[j][k] is a dot product of two rows.
  std::vector<double> Lt((size_t)m * m, 0.0);
  lower_inverse(L.data(), m, Lt.data(), true);

  // Gradient: pairs (i, j <= i) by rows, partial sums per chunk, added in chunk order.
  std::vector<double> part((size_t)kChunks * (d + 2), 0.0);
  parallel_chunks(kChunks, [&](int c) {
    double* g = part.data() + (size_t)c * (d + 2);
    for (int i = c; i < m; i += kChunks) {
      const double* ti = Lt.data() + (size_t)i * m;
      for (int j = 0; j <= i; ++j) {
        const double* tj = Lt.data() + (size_t)j * m;
        const double kinv = dot(ti + i, tj + i, m - i);
        const double Wij = alpha[i] * alpha[j] - kinv;
        const double mult = i == j ? 1.0 : 2.0;  // W and dK are symmetric
        double r2 = 0.0;
        double D2[SCOOT_MAX_DIM];
        for (int k = 0; k < d; ++k) {
          const double t = (X[(size_t)i * d + k] - X[(size_t)j * d + k]) * inv_ls[k];
          D2[k] = t * t;
          r2 += D2[k];
        }
        const double t = root * std::sqrt(r2);
        const double e = std::exp(-t);
        const double kf = m52 ? s2 * (1.0 + t + t * t / 3.0) * e : s2 * (1.0 + t) * e;
        const double radial = m52 ? 5.0 / 3.0 * s2 * (1.0 + t) * e : 3.0 * s2 * e;
        for (int k = 0; k < d; ++k) g[k] -= 0.5 * mult * Wij * radial * D2[k];
        g[d] -= 0.5 * mult * Wij * kf;
        if (i == j) g[d + 1] -= 0.5 * Wij * tau2;
      }
    }
  });
  for (int k = 0; k < d + 2; ++k) {
    double s = 0.0;
    for (int c = 0; c < kChunks; ++c) s += part[(size_t)c * (d + 2) + k];
    grad[k] = s;
  }
  return true;
}

int prepare(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
            const double* warp_b, double c, MleData& D) {
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
            const double* warp_b, double c, const double* theta, double* nll, double* grad) {
  if (!theta || !nll) return fail(SCOOT_ERR_INVALID_ARG, "gp nll: null pointer");
  MleData D;
  int rc = prepare(X, y, m, d, kernel, warp_a, warp_b, c, D);
  if (rc != SCOOT_OK) return rc;
  for (int k = 0; k < d + 2; ++k)
    if (!std::isfinite(theta[k])) return fail(SCOOT_ERR_INVALID_ARG, "gp nll: non-finite theta");
  if (!nll_eval(D, theta, nll, grad)) return fail(SCOOT_ERR_NOT_PD, "gp nll: K is not positive definite");
  return SCOOT_OK;
}

int mle_fit(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
            const double* warp_b, double c, const double* lower, const double* upper, int max_iter, double* theta,
            double* nll_out, int* iters_out) {
  if (!lower || !upper || !theta) return fail(SCOOT_ERR_INVALID_ARG, "gp mle: null pointer");
  if (max_iter < 1) return fail(SCOOT_ERR_INVALID_ARG, "gp mle: max_iter must be >= 1");
  MleData D;
  int rc = prepare(X, y, m, d, kernel, warp_a, warp_b, c, D);
  if (rc != SCOOT_OK) return rc;
  const int P = d + 2;
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
    if (!nll_eval(D, t.data(), &f, gth.data())) return false;
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
  to_theta(z, t);
  std::memcpy(theta, t.data(), sizeof(double) * P);
  if (nll_out) *nll_out = f;
  if (iters_out) *iters_out = it;
  return SCOOT_OK;
}

}  // namespace scoot
