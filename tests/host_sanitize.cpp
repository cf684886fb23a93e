// Host code of the library under the sanitizers: a CPU-only driver linked with
// the host sources (fit, Cholesky and inverse, likelihood search, forest
// training, EHVI boxes, forest packing, the thread pool), built once with
// AddressSanitizer + UndefinedBehaviorSanitizer and once with ThreadSanitizer
// by tests/test_host_sanitizers.py.  It exercises the paths the library's
// host tests reach, including searches and forest training run from several
// threads at once on the shared pool, and checks a few invariants (the
// factor reproduces K, the analytic gradient matches central differences,
// concurrent and sequential runs agree bit for bit).  Exit status 0 and no
// sanitizer report mean clean.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <string>
#include <thread>
#include <vector>

#include "internal.h"

namespace scoot {
// The library's error reporting lives with the C ABI (device code); the
// driver keeps its own copy.
namespace {
thread_local std::string g_err;
}
void clear_error() { g_err.clear(); }
void set_error(const std::string& msg) { g_err = msg; }
int fail(int status, const std::string& msg) {
  g_err = msg;
  return status;
}
int fail_static(int status, const char* msg) {
  g_err = msg;
  return status;
}
}  // namespace scoot

using namespace scoot;

static int g_bad = 0;
#define CHECK(cond, ...)                   \
  do {                                     \
    if (!(cond)) {                         \
      std::printf("FAIL: " __VA_ARGS__);   \
      std::printf("\n");                   \
      ++g_bad;                             \
    }                                      \
  } while (0)

struct Data {
  int m, d;
  std::vector<double> X, y;
};

static Data make_data(int m, int d, unsigned seed) {
  std::mt19937_64 rng(seed);
  std::uniform_real_distribution<double> u(0.0, 1.0);
  std::normal_distribution<double> nrm(0.0, 1.0);
  Data D{m, d, std::vector<double>((size_t)m * d), std::vector<double>(m)};
  for (auto& v : D.X) v = u(rng);
  for (int i = 0; i < m; ++i) {
    double s = 0;
    for (int k = 0; k < d; ++k) s += std::sin(3.0 * D.X[(size_t)i * d + k] * (k + 1));
    D.y[i] = s + 0.05 * nrm(rng);
  }
  return D;
}

static void check_cholesky_and_inverse() {
  const int m = 70;
  std::mt19937_64 rng(1);
  std::uniform_real_distribution<double> u(-1.0, 1.0);
  std::vector<double> B((size_t)m * m), A((size_t)m * m, 0.0);
  for (auto& v : B) v = u(rng);
  for (int i = 0; i < m; ++i)
    for (int j = 0; j < m; ++j) {
      double s = i == j ? m : 0.0;
      for (int k = 0; k < m; ++k) s += B[(size_t)i * m + k] * B[(size_t)j * m + k];
      A[(size_t)i * m + j] = s;
    }
  std::vector<double> L = A;
  CHECK(cholesky_lower(L.data(), m), "cholesky failed");
  double err = 0, scale = 0;
  for (int i = 0; i < m; ++i)
    for (int j = 0; j <= i; ++j) {
      double s = 0;
      for (int k = 0; k <= j; ++k) s += L[(size_t)i * m + k] * L[(size_t)j * m + k];
      err = std::fmax(err, std::fabs(s - A[(size_t)i * m + j]));
      scale = std::fmax(scale, std::fabs(A[(size_t)i * m + j]));
    }
  CHECK(err <= 1e-12 * scale, "L L^T != A (%g)", err);
  std::vector<double> Li((size_t)m * m), Lt((size_t)m * m);
  lower_inverse(L.data(), m, Li.data(), false);
  lower_inverse(L.data(), m, Lt.data(), true);
  double e2 = 0;
  for (int i = 0; i < m; ++i)
    for (int j = 0; j < m; ++j) {
      double s = 0;
      for (int k = 0; k < m; ++k) s += Li[(size_t)i * m + k] * L[(size_t)k * m + j];
      e2 = std::fmax(e2, std::fabs(s - (i == j ? 1.0 : 0.0)));
      CHECK(Li[(size_t)i * m + j] == Lt[(size_t)j * m + i], "transposed inverse differs at %d %d", i, j);
    }
  CHECK(e2 <= 1e-10, "L^-1 L != I (%g)", e2);
  // not positive definite
  std::vector<double> N((size_t)4 * 4, 0.0);
  N[0] = 1;
  N[5] = -1;
  CHECK(!cholesky_lower(N.data(), 4), "indefinite matrix factored");
}

static void check_fit() {
  for (int warped = 0; warped < 2; ++warped)
    for (scoot_kernel kern : {SCOOT_MATERN52, SCOOT_MATERN32}) {
      Data D = make_data(93, 7, 2 + warped);
      std::vector<double> ls(7, 0.4), wa(7, 1.3), wb(7, 0.8);
      FitHost f;
      const int rc = fit_host(D.X.data(), D.y.data(), D.m, D.d, kern, ls.data(), warped ? wa.data() : nullptr,
                              warped ? wb.data() : nullptr, 1.2, 1e-3, 0.1, f);
      CHECK(rc == SCOOT_OK, "fit_host rc %d", rc);
      std::vector<float> p32;
      std::vector<double> p64;
      pack_linv_f32(f, p32);
      pack_linv_f64(f, p64);
      CHECK(!p32.empty() && !p64.empty(), "empty packing");
    }
  // invalid inputs go through the error paths
  Data D = make_data(10, 3, 9);
  std::vector<double> ls = {0.5, -1.0, 0.5};
  FitHost f;
  CHECK(fit_host(D.X.data(), D.y.data(), D.m, D.d, SCOOT_MATERN52, ls.data(), nullptr, nullptr, 1.0, 1e-3, 0.0, f) !=
            SCOOT_OK,
        "negative lengthscale accepted");
}

static void check_nll_gradient() {
  for (int warped = 0; warped < 2; ++warped)
    for (scoot_kernel kern : {SCOOT_MATERN52, SCOOT_MATERN32}) {
      Data D = make_data(57, 4, 5 + warped);
      const int P = D.d + 2;
      std::vector<double> th = {std::log(0.3), std::log(0.7), std::log(0.5), std::log(1.1), std::log(1.4),
                                std::log(2e-3)};
      std::vector<double> wa = {1.5, 0.7, 1.0, 2.0}, wb = {0.6, 1.2, 1.0, 1.7};
      const double* pa = warped ? wa.data() : nullptr;
      const double* pb = warped ? wb.data() : nullptr;
      double f0, g[SCOOT_MAX_DIM + 2];
      CHECK(mle_nll(D.X.data(), D.y.data(), D.m, D.d, kern, pa, pb, 0.2, th.data(), &f0, g) == SCOOT_OK, "nll");
      for (int k = 0; k < P; ++k) {
        const double h = 1e-5;
        std::vector<double> tp = th, tm = th;
        tp[k] += h;
        tm[k] -= h;
        double fp, fm;
        mle_nll(D.X.data(), D.y.data(), D.m, D.d, kern, pa, pb, 0.2, tp.data(), &fp, nullptr);
        mle_nll(D.X.data(), D.y.data(), D.m, D.d, kern, pa, pb, 0.2, tm.data(), &fm, nullptr);
        const double fd = (fp - fm) / (2 * h);
        CHECK(std::fabs(fd - g[k]) <= 1e-5 * std::fmax(1.0, std::fabs(g[k])), "gradient %d: %g vs %g", k, g[k], fd);
      }
    }
}

struct MleRun {
  std::vector<double> theta;
  double nll = 0;
  int iters = 0, rc = 0;
};

static MleRun run_mle(const Data& D, int max_iter) {
  const int P = D.d + 2;
  MleRun r;
  r.theta.assign(P, 0.0);
  for (int k = 0; k < D.d; ++k) r.theta[k] = std::log(0.5);
  r.theta[D.d + 1] = std::log(1e-3);
  std::vector<double> lo(P), hi(P);
  for (int k = 0; k < D.d; ++k) {
    lo[k] = std::log(0.01);
    hi[k] = std::log(10.0);
  }
  lo[D.d] = std::log(0.05);
  hi[D.d] = std::log(20.0);
  lo[D.d + 1] = std::log(1e-6);
  hi[D.d + 1] = 0.0;
  r.rc = mle_fit(D.X.data(), D.y.data(), D.m, D.d, SCOOT_MATERN52, nullptr, nullptr, 0.0, lo.data(), hi.data(),
                 max_iter, r.theta.data(), &r.nll, &r.iters);
  return r;
}

static void check_concurrent_searches() {
  std::vector<Data> data = {make_data(120, 5, 11), make_data(96, 6, 12), make_data(80, 4, 13)};
  std::vector<MleRun> seq;
  for (const Data& D : data) seq.push_back(run_mle(D, 30));
  std::vector<MleRun> par(data.size());
  std::vector<std::thread> th;
  for (size_t i = 0; i < data.size(); ++i) th.emplace_back([&, i] { par[i] = run_mle(data[i], 30); });
  for (auto& t : th) t.join();
  for (size_t i = 0; i < data.size(); ++i) {
    CHECK(seq[i].rc == SCOOT_OK && par[i].rc == SCOOT_OK, "mle rc");
    CHECK(seq[i].nll == par[i].nll && seq[i].iters == par[i].iters, "concurrent search %zu differs", i);
    CHECK(std::memcmp(seq[i].theta.data(), par[i].theta.data(), seq[i].theta.size() * 8) == 0, "theta %zu", i);
  }
}

static void check_forest() {
  const int n = 300, d = 5;
  std::mt19937_64 rng(21);
  std::uniform_real_distribution<double> u(0.0, 1.0);
  std::vector<double> X((size_t)n * d), y(n);
  for (auto& v : X) v = u(rng);
  for (int i = 0; i < n; ++i) y[i] = (X[(size_t)i * d] + X[(size_t)i * d + 3] < 1.1) ^ (u(rng) < 0.05) ? 1.0 : 0.0;
  TrainedForest a, b;
  CHECK(train_forest_host(X.data(), y.data(), n, d, 12, 8, 77, true, a) == SCOOT_OK, "forest");
  std::thread t1([&] { train_forest_host(X.data(), y.data(), n, d, 12, 8, 77, true, b); });
  TrainedForest c;
  std::thread t2([&] { train_forest_host(X.data(), y.data(), n, d, 9, 6, 5, false, c); });
  t1.join();
  t2.join();
  CHECK(a.feature == b.feature && a.threshold == b.threshold && a.value == b.value && a.left == b.left,
        "forest training not reproducible across threads");
  // into the device format (host packing only)
  const size_t N = a.feature.size();
  std::vector<int32_t> feat(N), q16(N);
  std::vector<float> thr(N);
  for (size_t k = 0; k < N; ++k) {
    const bool leaf = a.left[k] < 0;
    feat[k] = leaf ? 0 : a.feature[k];
    float t = (float)a.threshold[k];
    if ((double)t > a.threshold[k]) t = std::nextafter(t, -INFINITY);
    thr[k] = leaf ? 0.0f : t;
    q16[k] = leaf ? (int32_t)std::nearbyint(a.value[k] * 65536.0) : 0;
  }
  ForestHost fh;
  CHECK(pack_forest(feat.data(), thr.data(), a.left.data(), a.right.data(), q16.data(), a.tree_offset.data(),
                    (int)a.tree_offset.size() - 1, d, fh) == SCOOT_OK,
        "pack_forest");
}

static void check_boxes() {
  std::mt19937_64 rng(31);
  std::uniform_real_distribution<double> u(0.0, 1.0);
  for (int p = 1; p <= 3; ++p)
    for (int m : {0, 1, 7, 60}) {
      std::vector<double> Y((size_t)m * p);
      for (int i = 0; i < m; ++i) {
        double s = 0;
        for (int j = 0; j < p; ++j) s += (Y[(size_t)i * p + j] = u(rng));
        for (int j = 0; j < p; ++j) Y[(size_t)i * p + j] /= s;  // on a simplex: many front points
      }
      std::vector<double> ref(p, 1.1);
      BoxTable bt;
      CHECK(build_boxes(m ? Y.data() : nullptr, m, p, ref.data(), bt) == SCOOT_OK, "boxes p=%d m=%d", p, m);
    }
}

static void check_pool() {
  std::vector<long long> out(1000, 0);
  for (int rep = 0; rep < 50; ++rep)
    parallel_chunks(37, [&](int c) {
      for (int i = c; i < 1000; i += 37) out[i] += i;
    });
  for (int i = 0; i < 1000; ++i) CHECK(out[i] == 50LL * i, "pool sum at %d", i);
  // several callers at once
  std::vector<std::thread> th;
  std::vector<long long> sums(4, 0);
  for (int t = 0; t < 4; ++t)
    th.emplace_back([&, t] {
      for (int rep = 0; rep < 20; ++rep) {
        std::vector<long long> part(16, 0);
        parallel_chunks(16, [&](int c) { part[c] = c + t; });
        for (long long v : part) sums[t] += v;
      }
    });
  for (auto& x : th) x.join();
  for (int t = 0; t < 4; ++t) CHECK(sums[t] == 20LL * (120 + 16 * t), "concurrent pool callers %d", t);
}

int main() {
  check_cholesky_and_inverse();
  check_fit();
  check_nll_gradient();
  check_concurrent_searches();
  check_forest();
  check_boxes();
  check_pool();
  std::printf("%s: %d failure(s)\n", g_bad ? "BAD" : "OK", g_bad);
  return g_bad ? 1 : 0;
}
