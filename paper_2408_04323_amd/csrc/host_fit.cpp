// Host side of the GP fit (Sec. 4.3, Eq. 4-5): K = k(X, X) + tau^2 I with a
// Matern ARD covariance (5/2, or the paper's 3/2) on optionally warped inputs,
// its Cholesky factor L, alpha = K^-1 (y - c), and the explicit inverse factor
// L^-1 that the device applies to k(X, x).
//
// Both covariances are s2 P(u) 2^-u in u = sqrt(2 nu) r log2(e): Matern-5/2
// has P = 1 + u ln2 + (u ln2)^2 / 3, Matern-3/2 has P = 1 + u ln2, so the
// device evaluates (coef0 + u (coef1 + u coef2)) 2^-u with per-dimension
// scales sqrt(2 nu) log2(e) / l_k folded into the coordinates.
//
// sigma^2(x) = s2 - ||L^-1 k(X, x)||^2, so the device needs L^-1 (lower
// triangular).  Applying it as a triangular matrix product instead of a
// substitution removes every dependency between row blocks, so all row blocks
// of a candidate tile can run on the matrix cores at once.
#include <cmath>
#include <cstring>
#include <string>

#include "internal.h"

namespace scoot {

namespace {
constexpr double kSqrt5 = 2.23606797749978969641;
constexpr double kSqrt3 = 1.73205080756887729353;
constexpr double kLog2e = 1.44269504088896340736;
constexpr double kLn2 = 0.69314718055994530942;

bool finite_all(const double* v, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!std::isfinite(v[i])) return false;
  return true;
}
}  // namespace

int fit_setup(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* ls,
              const double* warp_a, const double* warp_b, double s2, double tau2, double c, FitHost& f) {
  if (!X || !y || !ls) return fail(SCOOT_ERR_INVALID_ARG, "gp fit: null pointer");
  if (kernel != SCOOT_MATERN52 && kernel != SCOOT_MATERN32) return fail(SCOOT_ERR_INVALID_ARG, "gp fit: bad kernel");
  if ((warp_a == nullptr) != (warp_b == nullptr))
    return fail(SCOOT_ERR_INVALID_ARG, "gp fit: warp_a and warp_b go together");
  if (m < 1 || d < 1) return fail(SCOOT_ERR_INVALID_ARG, "gp fit: m and d must be >= 1");
  if (d > SCOOT_MAX_DIM) return fail(SCOOT_ERR_UNSUPPORTED, "gp fit: d exceeds SCOOT_MAX_DIM");
  if (m > SCOOT_MAX_OBS) return fail(SCOOT_ERR_UNSUPPORTED, "gp fit: m exceeds SCOOT_MAX_OBS");
  if (!finite_all(X, (size_t)m * d) || !finite_all(y, m))
    return fail(SCOOT_ERR_INVALID_ARG, "gp fit: non-finite observation");
  for (int k = 0; k < d; ++k)
    if (!(ls[k] > 0) || !std::isfinite(ls[k]))
      return fail(SCOOT_ERR_INVALID_ARG, "gp fit: lengthscales must be finite and > 0");
  if (!(s2 > 0) || !std::isfinite(s2) || !(tau2 >= 0) || !std::isfinite(tau2) || !std::isfinite(c))
    return fail(SCOOT_ERR_INVALID_ARG, "gp fit: bad signal/noise variance or prior mean");

  if (warp_a)
    for (int k = 0; k < d; ++k)
      if (!(warp_a[k] > 0) || !(warp_b[k] > 0) || !std::isfinite(warp_a[k]) || !std::isfinite(warp_b[k]))
        return fail(SCOOT_ERR_INVALID_ARG, "gp fit: warping parameters must be finite and > 0");

  f.m = m;
  f.d = d;
  f.kernel = kernel;
  f.m_pad = (m + kBlk32 - 1) / kBlk32 * kBlk32;
  f.nb = f.m_pad / kBlk32;
  f.s2 = s2;
  f.tau2 = tau2;
  f.c = c;
  const double root = kernel == SCOOT_MATERN52 ? kSqrt5 : kSqrt3;  // sqrt(2 nu)
  f.coef[0] = s2;
  f.coef[1] = s2 * kLn2;
  f.coef[2] = kernel == SCOOT_MATERN52 ? s2 * kLn2 * kLn2 / 3.0 : 0.0;
  f.scale.assign(d, 0.0);
  for (int k = 0; k < d; ++k) f.scale[k] = root * kLog2e / ls[k];
  f.Xw.assign(X, X + (size_t)m * d);
  if (warp_a) {
    f.warp_a.assign(warp_a, warp_a + d);
    f.warp_b.assign(warp_b, warp_b + d);
    for (int i = 0; i < m; ++i)
      for (int k = 0; k < d; ++k) f.Xw[(size_t)i * d + k] = kumaraswamy(X[(size_t)i * d + k], warp_a[k], warp_b[k]);
  }
  return SCOOT_OK;
}

int fit_host(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* ls,
             const double* warp_a, const double* warp_b, double s2, double tau2, double c, FitHost& f) {
  const int rc = fit_setup(X, y, m, d, kernel, ls, warp_a, warp_b, s2, tau2, c, f);
  if (rc != SCOOT_OK) return rc;
  const double root = kernel == SCOOT_MATERN52 ? kSqrt5 : kSqrt3;  // sqrt(2 nu)
  std::vector<double> inv_ls(d);
  for (int k = 0; k < d; ++k) inv_ls[k] = 1.0 / ls[k];

  // K = k(X, X) + tau^2 I (lower triangle; rows in parallel), factored in place.
  f.L.assign((size_t)m * m, 0.0);
  double* L = f.L.data();
  const double* Xw = f.Xw.data();
  constexpr int kChunks = 32;
  parallel_chunks(kChunks, [&](int ch) {
    for (int i = ch; i < m; i += kChunks)
      for (int j = 0; j <= i; ++j) {
        double r2 = 0;
        for (int k = 0; k < d; ++k) {
          double t = (Xw[(size_t)i * d + k] - Xw[(size_t)j * d + k]) * inv_ls[k];
          r2 += t * t;
        }
        const double t = root * std::sqrt(r2);
        const double kv = kernel == SCOOT_MATERN52 ? s2 * (1.0 + t + t * t / 3.0) * std::exp(-t)
                                                   : s2 * (1.0 + t) * std::exp(-t);
        L[(size_t)i * m + j] = kv + (i == j ? tau2 : 0.0);
      }
  });
  // L L^T = K.  A pivot that is not positive, or below 1e-13 of its diagonal
  // entry, means K is not numerically positive definite.
  if (!cholesky_lower(L, m)) return fail(SCOOT_ERR_NOT_PD, "gp fit: K + tau^2 I is not positive definite");

  // alpha = L^-T L^-1 (y - c).
  std::vector<double> z(m);
  for (int i = 0; i < m; ++i) {
    double dot = 0.0;
#pragma omp simd reduction(+ : dot)
    for (int k = 0; k < i; ++k) dot += L[(size_t)i * m + k] * z[k];
    double s = y[i] - c - dot;
    z[i] = s / L[(size_t)i * m + i];
  }
  f.alpha.assign(m, 0.0);
  for (int i = m - 1; i >= 0; --i) {
    double s = z[i];
    for (int k = i + 1; k < m; ++k) s -= L[(size_t)k * m + i] * f.alpha[k];
    f.alpha[i] = s / L[(size_t)i * m + i];
  }

  // L^-1 column by column: forward substitution of L w = e_j.
  f.Linv.assign((size_t)m * m, 0.0);
  lower_inverse(L, m, f.Linv.data(), false);
  return SCOOT_OK;
}

// fp32 layout, for v_mfma_f32_16x16x4f32: 16 x 16 blocks (J <= I), the
// block's contraction index ordered k = 4g + s (g = lane / 16, s the step),
// so at step s lane l holds Linv[16I + l % 16][16J + 4 (l / 16) + s] and a
// lane reads the four steps of a block as one 16-byte load:
//   float index = (blk * 64 + l) * 4 + s.
// Blocks are ordered the way the kernel's waves consume them: plan entry
// after plan entry (plan_rows16 with the kernel's wave count), J = 0..I.
void pack_linv_f32(const FitHost& f, std::vector<float>& out) {
  const int nb = f.m_pad / kBlk16, m = f.m;
  const RowPlan16 plan = plan_rows16(nb, posterior_waves(f.nb));
  out.assign((size_t)nb * (nb + 1) / 2 * 4 * 64, 0.0f);
  size_t blk = 0;
  for (int e = 0; e < 8; ++e)
    for (int q = 0; q < plan.nrows[e] && q < kMaxRows16; ++q) {
      const int I = plan16_row(plan, e, q);
      for (int J = 0; J <= I; ++J, ++blk)
        for (int l = 0; l < 64; ++l)
          for (int s = 0; s < 4; ++s) {
            const int row = 16 * I + (l % 16), col = 16 * J + 4 * (l / 16) + s;
            const double v = (row < m && col < m) ? f.Linv[(size_t)row * m + col] : 0.0;
            out[(blk * 64 + l) * 4 + s] = (float)v;
          }
    }
}

// The fp32 kernel's observation operand: per 16-observation block J and step
// s of a v_mfma_f64_16x16x4f64 chain, lane l holds component k = 4s + l / 16
// of an observation's augmented row (2 Xs_i, -|Xs_i|^2, -1, 0 ...) (Xs the
// warped inputs times the per-dimension scales), so that with the
// candidates' rows (xs, 1, |xs|^2) the chain yields -|xs - Xs_i|^2:
//   double index = (J * S + s) * 64 + l,  S = ceil((d + 2) / 4).
// That instruction leaves output row t = g + 4r in register r of lanes
// 16g .. 16g + 15 (measured), while the float triangle wants observation
// 16J + 4g + r there, so A-operand row t carries observation
// 16J + 4 (t % 4) + t / 4.  Padding rows (i >= m) carry -1e30 in the norm's
// place: their covariance underflows to exactly 0.
void pack_obs_f32(const FitHost& f, std::vector<double>& out) {
  const int nb = f.m_pad / kBlk16, m = f.m, d = f.d, S = (d + 2 + 3) / 4;
  out.assign((size_t)nb * S * 64, 0.0);
  for (int J = 0; J < nb; ++J)
    for (int s = 0; s < S; ++s)
      for (int l = 0; l < 64; ++l) {
        const int t = l % 16, i = 16 * J + 4 * (t % 4) + t / 4, k = 4 * s + l / 16;
        double v = 0.0;
        if (i < m) {
          if (k < d) {
            v = 2.0 * f.Xw[(size_t)i * d + k] * f.scale[k];
          } else if (k == d) {
            double nrm = 0.0;
            for (int q = 0; q < d; ++q) {
              const double t = f.Xw[(size_t)i * d + q] * f.scale[q];
              nrm += t * t;
            }
            v = -nrm;
          } else if (k == d + 1) {
            v = -1.0;
          }
        } else {
          v = k == d ? -1e30 : (k == d + 1 ? -1.0 : 0.0);
        }
        out[((size_t)J * S + s) * 64 + l] = v;
      }
}

// fp64 layout, for v_mfma_f64_16x16x4f64: 16 x 16 blocks, four steps per
// block; at step s lane l holds Linv[16I + l % 16][16J + 4s + l / 16]; steps
// are paired so a lane reads two consecutive steps as one 16-byte load:
//   double index = ((blk * 2 + s / 2) * 64 + l) * 2 + s % 2.
// Blocks are ordered as for fp32: plan entry after plan entry, J = 0..I.
void pack_linv_f64(const FitHost& f, std::vector<double>& out) {
  const int nb = f.m_pad / kBlk16, m = f.m;
  const RowPlan16 plan = plan_rows16(nb, posterior_waves(f.nb));
  out.assign((size_t)nb * (nb + 1) / 2 * 4 * 64, 0.0);
  size_t blk = 0;
  for (int e = 0; e < 8; ++e)
    for (int q = 0; q < plan.nrows[e] && q < kMaxRows16; ++q) {
      const int I = plan16_row(plan, e, q);
      for (int J = 0; J <= I; ++J, ++blk)
        for (int s = 0; s < 4; ++s)
          for (int l = 0; l < 64; ++l) {
            int r = 16 * I + (l % 16), col = 16 * J + 4 * s + l / 16;
            double v = (r < m && col < m) ? f.Linv[(size_t)r * m + col] : 0.0;
            out[((blk * 2 + s / 2) * 64 + l) * 2 + s % 2] = v;
          }
    }
}

}  // namespace scoot
