// The suggestion step end to end (Algorithm 1's SUGGEST; Sec. 4.1 steps
// 3-6): standardise the valid observations, learn each objective's GP
// hyperparameters by maximum likelihood (Sec. 4.3), fit the GPs, train the
// feasibility forest on every observation (Sec. 4.7), generate the Sobol pool
// with its known-constraint mask (Sec. 4.5.3), score it -- MACE for one
// objective (Sec. 4.5.1), EHVI top-k for several (Sec. 4.5.2) -- under
// POF >= Delta (Eq. 3), and fill a shortfall with admissible Sobol points
// (Sec. 4.7, last paragraph).  Built on the library's own entry points; the
// pool and every score stay on the device, only k indices come back.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <new>
#include <string>
#include <system_error>
#include <thread>
#include <vector>

#include "internal.h"

namespace scoot {
namespace {

constexpr double kDefaultLo[3] = {0.01, 0.05, 1e-6};   // lengthscale, signal var, noise var
constexpr double kDefaultHi[3] = {10.0, 20.0, 1.0};
constexpr double kDefaultStart[3] = {0.5, 1.0, 1e-3};
constexpr double kWarpLo = 0.2, kWarpHi = 5.0;         // box of each learned Kumaraswamy parameter
constexpr int kDefaultMleIter = 200;

// With the warping learned: the box and start of the warp parameters (log a,
// then log b), after the d + 2 of theta_box; the start is the caller's fixed
// warp when given, else the identity a = b = 1.
void warp_box(const scoot_suggest_opts& o, int j, int d, double* lo, double* hi, double* th) {
  for (int t = 0; t < 2 * d; ++t) {
    lo[t] = std::log(kWarpLo);
    hi[t] = std::log(kWarpHi);
    const double* w = t < d ? o.warp_a : o.warp_b;
    th[t] = w ? std::log(w[(size_t)j * d + t % d]) : 0.0;
    th[t] = std::fmin(std::fmax(th[t], lo[t]), hi[t]);
  }
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

// Box and start of objective j's likelihood search: the caller's, else the defaults.
void theta_box(const scoot_suggest_opts& o, int j, int d, double* lo, double* hi, double* th) {
  const int nt = d + 2;
  for (int t = 0; t < nt; ++t) {
    const int kind = t < d ? 0 : t - d + 1;
    lo[t] = o.theta_lower ? o.theta_lower[(size_t)j * nt + t] : std::log(kDefaultLo[kind]);
    hi[t] = o.theta_upper ? o.theta_upper[(size_t)j * nt + t] : std::log(kDefaultHi[kind]);
    th[t] = o.theta_start ? o.theta_start[(size_t)j * nt + t] : std::log(kDefaultStart[kind]);
    th[t] = std::fmin(std::fmax(th[t], lo[t]), hi[t]);
  }
}

// Releases the handles a call creates, whatever path it leaves by.
struct Handles {
  std::vector<scoot_gp> gps;
  scoot_forest forest = nullptr;
  ~Handles() {
    for (scoot_gp g : gps) scoot_gp_destroy(g);
    if (forest) scoot_forest_destroy(forest);
  }
};

bool finite_all(const double* v, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!std::isfinite(v[i])) return false;
  return true;
}

int check_space(const scoot_space* sp) {
  if (!sp) return fail(SCOOT_ERR_INVALID_ARG, "suggest: null space");
  if (sp->d < 1 || sp->d > SCOOT_MAX_DIM) return fail(SCOOT_ERR_INVALID_ARG, "suggest: d out of range");
  if (!sp->levels || !sp->sobol_poly || !sp->sobol_vinit) return fail(SCOOT_ERR_INVALID_ARG, "suggest: null space table");
  if (sp->r < 0) return fail(SCOOT_ERR_INVALID_ARG, "suggest: r < 0");
  if (sp->r > 0 && (!sp->A || !sp->b)) return fail(SCOOT_ERR_INVALID_ARG, "suggest: null constraint rows");
  return SCOOT_OK;
}

int check_opts(const scoot_suggest_opts* o, int p, int d) {
  if (!o) return fail(SCOOT_ERR_INVALID_ARG, "suggest: null opts");
  if (o->k < 1 || o->k > SCOOT_MAX_Q) return fail(SCOOT_ERR_INVALID_ARG, "suggest: k out of range");
  if (!(o->delta >= 0.0 && o->delta <= 1.0)) return fail(SCOOT_ERR_INVALID_ARG, "suggest: delta outside [0, 1]");
  if (o->pool_size < 1 || o->pool_size >= ((int64_t)1 << 31))
    return fail(SCOOT_ERR_INVALID_ARG, "suggest: pool_size out of range");
  if (o->pool_skip < 0) return fail(SCOOT_ERR_INVALID_ARG, "suggest: pool_skip < 0");
  if (o->kernel != SCOOT_MATERN52 && o->kernel != SCOOT_MATERN32)
    return fail(SCOOT_ERR_INVALID_ARG, "suggest: unknown kernel");
  if (o->dtype != SCOOT_F32 && o->dtype != SCOOT_F64) return fail(SCOOT_ERR_INVALID_ARG, "suggest: unknown dtype");
  if ((o->warp_a == nullptr) != (o->warp_b == nullptr))
    return fail(SCOOT_ERR_INVALID_ARG, "suggest: warp_a and warp_b go together");
  if (o->learn_warp != 0 && o->learn_warp != 1) return fail(SCOOT_ERR_INVALID_ARG, "suggest: learn_warp is 0 or 1");
  if (o->warp_a)
    for (size_t t = 0; t < (size_t)p * d; ++t)
      if (!(o->warp_a[t] > 0) || !(o->warp_b[t] > 0) || !std::isfinite(o->warp_a[t]) || !std::isfinite(o->warp_b[t]))
        return fail(SCOOT_ERR_INVALID_ARG, "suggest: warping parameters must be finite and > 0");
  if (o->n_trees < 1 || o->n_trees > SCOOT_MAX_TREES) return fail(SCOOT_ERR_INVALID_ARG, "suggest: n_trees out of range");
  if (o->max_depth < 0) return fail(SCOOT_ERR_INVALID_ARG, "suggest: max_depth < 0");
  if (!std::isfinite(o->xi)) return fail(SCOOT_ERR_INVALID_ARG, "suggest: non-finite xi");
  if (p == 1 && o->t < 1) return fail(SCOOT_ERR_INVALID_ARG, "suggest: t < 1");
  const size_t nt = (size_t)p * (d + 2);
  for (const double* v : {o->theta_lower, o->theta_upper, o->theta_start})
    if (v && !finite_all(v, nt)) return fail(SCOOT_ERR_INVALID_ARG, "suggest: non-finite hyperparameter bound");
  if (o->ref && !finite_all(o->ref, (size_t)p)) return fail(SCOOT_ERR_INVALID_ARG, "suggest: non-finite ref");
  for (int j = 0; j < p; ++j) {
    double lo[SCOOT_MAX_DIM + 2], hi[SCOOT_MAX_DIM + 2], th[SCOOT_MAX_DIM + 2];
    theta_box(*o, j, d, lo, hi, th);
    for (int t = 0; t < d + 2; ++t)
      if (!(lo[t] <= hi[t])) return fail(SCOOT_ERR_INVALID_ARG, "suggest: theta_lower above theta_upper");
  }
  return SCOOT_OK;
}

}  // namespace
}  // namespace scoot

using namespace scoot;

int scoot_suggest(const double* X_obs, const double* Y_obs, const uint8_t* valid, int n_obs, int p,
                  const scoot_space* space, const scoot_suggest_opts* opts, double* x_out, int32_t* source,
                  double* theta_out, int* n_out, void* stream) {
  set_error("");
  int rc = check_space(space);
  if (rc != SCOOT_OK) return rc;
  const int d = space->d;
  if (p < 1 || p > SCOOT_MAX_OBJECTIVES) return fail(SCOOT_ERR_INVALID_ARG, "suggest: p out of range");
  rc = check_opts(opts, p, d);
  if (rc != SCOOT_OK) return rc;
  if (n_obs < 0 || (n_obs > 0 && (!X_obs || !Y_obs || !valid)))
    return fail(SCOOT_ERR_INVALID_ARG, "suggest: bad observations");
  if (!x_out || !n_out) return fail(SCOOT_ERR_INVALID_ARG, "suggest: null output");
  if (!finite_all(X_obs, (size_t)n_obs * d)) return fail(SCOOT_ERR_INVALID_ARG, "suggest: non-finite X_obs");
  const scoot_suggest_opts& o = *opts;
  const int k = o.k;
  const int64_t n = o.pool_size;
  hipStream_t s = (hipStream_t)stream;
  try {
    // ---- 1. valid observations, standardised per objective -------------
    std::vector<int> rows;
    for (int i = 0; i < n_obs; ++i)
      if (valid[i]) rows.push_back(i);
    const int m = (int)rows.size();
    if (m > SCOOT_MAX_OBS) return fail(SCOOT_ERR_UNSUPPORTED, "suggest: more valid observations than SCOOT_MAX_OBS");
    std::vector<double> Xv((size_t)m * d), Yv((size_t)m * p), mean(p, 0.0), scale(p, 1.0);
    for (int r = 0; r < m; ++r) {
      std::memcpy(&Xv[(size_t)r * d], X_obs + (size_t)rows[r] * d, sizeof(double) * d);
      for (int j = 0; j < p; ++j) Yv[(size_t)r * p + j] = Y_obs[(size_t)rows[r] * p + j];
    }
    if (!finite_all(Yv.data(), Yv.size())) return fail(SCOOT_ERR_INVALID_ARG, "suggest: non-finite valid Y_obs");
    for (int j = 0; j < p && m > 0; ++j) {
      double sum = 0.0;
      for (int r = 0; r < m; ++r) sum += Yv[(size_t)r * p + j];
      mean[j] = sum / m;
      double ss = 0.0;
      for (int r = 0; r < m; ++r) {
        const double e = Yv[(size_t)r * p + j] - mean[j];
        ss += e * e;
      }
      const double sd = std::sqrt(ss / m);
      scale[j] = sd > 0.0 ? sd : 1.0;
      for (int r = 0; r < m; ++r) Yv[(size_t)r * p + j] = (Yv[(size_t)r * p + j] - mean[j]) / scale[j];
    }

    // ---- device scratch: pool, known mask, every score of the pass -------
    const size_t esz = o.dtype == SCOOT_F32 ? 4 : 8;
    size_t off = 0;
    auto take = [&](size_t bytes) {
      const size_t at = off;
      off += align256(bytes);
      return at;
    };
    const size_t o_xc = take((size_t)n * d * 4), o_known = take((size_t)n), o_mu = take((size_t)p * n * esz),
                 o_sd = take((size_t)p * n * esz), o_s1 = take((size_t)n * esz), o_s2 = take((size_t)n * esz),
                 o_s3 = take((size_t)n * esz), o_votes = take((size_t)n * 4), o_mask = take((size_t)n),
                 o_front = take((size_t)n), o_idx = take((size_t)k * 8), o_cnt = take(16), o_sc = take((size_t)k * 8);
    unsigned char* ws = (unsigned char*)device_scratch(off, 6);
    if (!ws) return fail(SCOOT_ERR_NO_MEMORY, "suggest: scratch allocation failed");
    float* Xc = (float*)(ws + o_xc);
    uint8_t* known = ws + o_known;
    int64_t* idx_dev = (int64_t*)(ws + o_idx);

    // ---- 4. pool and known constraints ---------------------------------
    rc = scoot_sobol_pool(space->sobol_poly, space->sobol_vinit, d, space->levels, o.pool_skip, n, space->A,
                          space->b, space->r, Xc, known, stream);
    if (rc != SCOOT_OK) return rc;

    std::vector<int64_t> picked;
    Handles h;
    if (m > 0) {
      // ---- 2. hyperparameters and GPs ----------------------------------
      // theta per objective: d + 2 entries, or 3d + 2 with the warping learned
      const bool lw = o.learn_warp != 0;
      const int nt = lw ? 3 * d + 2 : d + 2;
      std::vector<double> theta((size_t)p * nt);
      // The objectives' searches run side by side, each on its own thread and
      // each spreading its likelihood evaluations over the library's host
      // threads; every search is deterministic, so the result is the same as
      // one after the other.
      std::vector<int> search_rc(p, SCOOT_OK);
      std::vector<std::string> search_err(p);
      // Device searches: each objective's evaluations on a stream of its own,
      // so the objectives' kernels run side by side.
      const bool on_device = o.host_search == 0;
      int device = 0;
      if (hipGetDevice(&device) != hipSuccess) return fail(SCOOT_ERR_DEVICE, "suggest: no current device");
      std::vector<hipStream_t> streams(p, nullptr);
      h.gps.assign(p, nullptr);  // each search thread fits its objective's GP as soon as it has theta
      if (on_device) {
        for (int j = 0; j < p; ++j)
          if (hipStreamCreateWithFlags(&streams[j], hipStreamNonBlocking) != hipSuccess) {
            for (int q = 0; q < j; ++q) (void)hipStreamDestroy(streams[q]);
            return fail(SCOOT_ERR_DEVICE, "suggest: cannot create a stream");
          }
      }
      auto search = [&](int j) {
        try {
          double lo[3 * SCOOT_MAX_DIM + 2], hi[3 * SCOOT_MAX_DIM + 2], th[3 * SCOOT_MAX_DIM + 2];
          theta_box(o, j, d, lo, hi, th);
          if (lw) warp_box(o, j, d, lo + d + 2, hi + d + 2, th + d + 2);
          bool all_fixed = true;
          for (int t = 0; t < nt; ++t) all_fixed = all_fixed && lo[t] == hi[t];
          std::vector<double> yj(m);
          for (int r = 0; r < m; ++r) yj[r] = Yv[(size_t)r * p + j];
          const double* wa = o.warp_a ? o.warp_a + (size_t)j * d : nullptr;
          const double* wb = o.warp_b ? o.warp_b + (size_t)j * d : nullptr;
          const int iters = o.mle_max_iter > 0 ? o.mle_max_iter : kDefaultMleIter;
          if (hipSetDevice(device) != hipSuccess) {
            search_rc[j] = SCOOT_ERR_DEVICE;
            search_err[j] = "suggest: cannot select the device";
            return;
          }
          if (!all_fixed && on_device) {
            // the search, then the GP at its optimum from the search's own
            // device factorization (no host refit)
            search_rc[j] = mle_fit_device_gp(Xv.data(), yj.data(), m, d, (scoot_kernel)o.kernel, lw ? nullptr : wa,
                                             lw ? nullptr : wb, 0.0, lw, lo, hi, iters, th, (scoot_dtype)o.dtype,
                                             streams[j], &h.gps[j]);
            if (search_rc[j] != SCOOT_OK) search_err[j] = scoot_last_error();  // this thread's message
            std::memcpy(&theta[(size_t)j * nt], th, sizeof(double) * nt);
            return;
          } else if (!all_fixed) {
            search_rc[j] = lw ? scoot_gp_mle_warp(Xv.data(), yj.data(), m, d, (scoot_kernel)o.kernel, 0.0, lo, hi,
                                                  iters, th, nullptr, nullptr)
                              : scoot_gp_mle(Xv.data(), yj.data(), m, d, (scoot_kernel)o.kernel, wa, wb, 0.0, lo,
                                             hi, iters, th, nullptr, nullptr);
            if (search_rc[j] != SCOOT_OK) search_err[j] = scoot_last_error();  // this thread's message
          }
          std::memcpy(&theta[(size_t)j * nt], th, sizeof(double) * nt);
          if (search_rc[j] != SCOOT_OK) return;
          // the GP at the hyperparameters found
          double ell[SCOOT_MAX_DIM], la[SCOOT_MAX_DIM], lb[SCOOT_MAX_DIM];
          for (int t = 0; t < d; ++t) ell[t] = std::exp(th[t]);
          if (lw) {
            for (int t = 0; t < d; ++t) {
              la[t] = std::exp(th[d + 2 + t]);
              lb[t] = std::exp(th[2 * d + 2 + t]);
            }
            wa = la;
            wb = lb;
          }
          // the fit's host steps leave a core to each search still running
          PoolHelpers cap(on_device ? std::max(0, (pool_threads() - p) / p - 1) : -1);
          search_rc[j] = scoot_gp_fit_ex(Xv.data(), yj.data(), m, d, (scoot_kernel)o.kernel, ell, wa, wb,
                                         std::exp(th[d]), std::exp(th[d + 1]), 0.0, (scoot_dtype)o.dtype, stream,
                                         &h.gps[j]);
          if (search_rc[j] != SCOOT_OK) search_err[j] = scoot_last_error();
        } catch (...) {
          search_rc[j] = SCOOT_ERR_NO_MEMORY;
          search_err[j] = "suggest: hyperparameter search ran out of memory";
        }
      };
      std::vector<std::thread> searches;
      searches.reserve(p);  // no reallocation once a thread runs
      // Device searches leave this thread free: it trains the forest meanwhile
      // (step 3, host work that does not depend on the hyperparameters).
      for (int j = on_device ? 0 : 1; j < p; ++j) {
        try {
          searches.emplace_back(search, j);
        } catch (const std::system_error&) {
          search(j);  // no thread to spare: run it here
        }
      }
      if (!on_device) search(0);
      // ---- 3. feasibility forest on every observation ---------------------
      std::vector<double> label(n_obs);
      for (int i = 0; i < n_obs; ++i) label[i] = valid[i] ? 1.0 : 0.0;
      int forest_rc;
      {
        // beside device searches, whose threads mostly launch and wait, the
        // forest leaves them a core each
        PoolHelpers cap(on_device ? std::max(0, pool_threads() - 1 - p) : -1);
        forest_rc = scoot_forest_train_create(X_obs, label.data(), n_obs, d, o.n_trees, o.max_depth, o.forest_seed,
                                              o.bootstrap, &h.forest);
      }
      const std::string forest_err = forest_rc != SCOOT_OK ? scoot_last_error() : "";
      for (auto& t : searches) t.join();
      for (hipStream_t st : streams)
        if (st) (void)hipStreamDestroy(st);
      if (forest_rc != SCOOT_OK) return fail(forest_rc, forest_err);
      for (int j = 0; j < p; ++j)
        if (search_rc[j] != SCOOT_OK) return fail(search_rc[j], search_err[j]);
      if (theta_out) std::memcpy(theta_out, theta.data(), sizeof(double) * theta.size());

      // ---- 5. score the pool and pick ----------------------------------
      void* mu = ws + o_mu;
      void* sd = ws + o_sd;
      int32_t* votes = (int32_t*)(ws + o_votes);
      uint8_t* mask = ws + o_mask;
      int32_t* cnt = (int32_t*)(ws + o_cnt);
      if (p == 1) {
        double best = Yv[0];
        for (int r = 1; r < m; ++r) best = std::fmin(best, Yv[r]);
        double beta = 0.0;
        rc = scoot_ucb_beta(o.t, &beta);
        if (rc != SCOOT_OK) return rc;
        rc = scoot_suggest_mace_ex(h.gps[0], h.forest, known, Xc, n, best, o.xi, beta, o.delta, o.pick_seed, k, mu,
                                   sd, ws + o_s1, ws + o_s2, ws + o_s3, votes, mask, ws + o_front, idx_dev, cnt,
                                   stream);
      } else {
        double ref[SCOOT_MAX_OBJECTIVES];
        for (int j = 0; j < p; ++j) {
          if (o.ref) {
            ref[j] = (o.ref[j] - mean[j]) / scale[j];
          } else {
            double lo = Yv[j], hi = Yv[j];
            for (int r = 1; r < m; ++r) {
              lo = std::fmin(lo, Yv[(size_t)r * p + j]);
              hi = std::fmax(hi, Yv[(size_t)r * p + j]);
            }
            ref[j] = hi + 0.1 * (hi - lo);
          }
        }
        rc = scoot_score_pool_ex(h.gps.data(), p, h.forest, known, Xc, n, 0.0, 0.0, Yv.data(), m, ref, o.delta, k,
                                 mu, sd, ws + o_s1, votes, mask, idx_dev, ws + o_sc, cnt, stream);
      }
      if (rc != SCOOT_OK) return rc;
      int64_t idx_host[SCOOT_MAX_Q];
      if (hipMemcpyAsync(idx_host, idx_dev, sizeof(int64_t) * k, hipMemcpyDeviceToHost, s) != hipSuccess ||
          hipStreamSynchronize(s) != hipSuccess)
        return fail(SCOOT_ERR_DEVICE, "suggest: reading the picks back failed");
      for (int r = 0; r < k; ++r)
        if (idx_host[r] >= 0) picked.push_back(idx_host[r]);
    } else if (theta_out) {
      for (size_t t = 0; t < (size_t)p * (o.learn_warp ? 3 * d + 2 : d + 2); ++t) theta_out[t] = NAN;
    }
    const int n_solver = (int)picked.size();

    // ---- 6. Sobol fill ----------------------------------------------------
    if ((int)picked.size() < k) {
      std::vector<uint8_t> kh((size_t)n);
      if (hipMemcpyAsync(kh.data(), known, (size_t)n, hipMemcpyDeviceToHost, s) != hipSuccess ||
          hipStreamSynchronize(s) != hipSuccess)
        return fail(SCOOT_ERR_DEVICE, "suggest: reading the known mask back failed");
      std::vector<uint8_t> taken((size_t)n, 0);
      for (int64_t i : picked) taken[(size_t)i] = 1;
      for (int64_t i = 0; i < n && (int)picked.size() < k; ++i)
        if (kh[(size_t)i] && !taken[(size_t)i]) picked.push_back(i);
    }

    // ---- outputs -----------------------------------------------------------
    std::vector<float> row((size_t)d);
    for (size_t r = 0; r < picked.size(); ++r) {
      if (hipMemcpyAsync(row.data(), Xc + (size_t)picked[r] * d, sizeof(float) * d, hipMemcpyDeviceToHost, s) !=
              hipSuccess ||
          hipStreamSynchronize(s) != hipSuccess)
        return fail(SCOOT_ERR_DEVICE, "suggest: reading a configuration back failed");
      for (int t = 0; t < d; ++t) x_out[r * d + t] = (double)row[t];
      if (source) source[r] = (int)r < n_solver ? 0 : 1;
    }
    *n_out = (int)picked.size();
    return SCOOT_OK;
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "suggest: host allocation failed");
  }
}
