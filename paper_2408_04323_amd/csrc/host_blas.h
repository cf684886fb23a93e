// Register-blocked inner products for the host's dense fp64 steps (Cholesky
// factor, inverse factor, K^-1 in the likelihood gradient).  Every sum has a
// fixed order that depends only on its length and on whether the CPU has
// AVX2 (k mod 2 or k mod 4 accumulate in the lanes of a vector, the lanes are
// added at the end, then the last terms), so results do not depend on how
// work is split over threads.
#pragma once

#include <cstring>

#include <immintrin.h>

namespace scoot {

typedef double v2d __attribute__((vector_size(16)));

inline v2d load2(const double* p) {
  v2d v;
  std::memcpy(&v, p, sizeof v);
  return v;
}

// out[r][c] = sum_{k < n} a[r][k] * b[c][k], two lanes (baseline x86-64).
template <int R, int C>
inline void dots_tile_sse2(const double* const (&a)[R], const double* const (&b)[C], int n, double (&out)[R][C]) {
  v2d acc[R][C];
  for (int r = 0; r < R; ++r)
    for (int c = 0; c < C; ++c) acc[r][c] = v2d{0.0, 0.0};
  int k = 0;
  for (; k + 2 <= n; k += 2) {
    v2d av[R], bv[C];
    for (int r = 0; r < R; ++r) av[r] = load2(a[r] + k);
    for (int c = 0; c < C; ++c) bv[c] = load2(b[c] + k);
    for (int r = 0; r < R; ++r)
      for (int c = 0; c < C; ++c) acc[r][c] += av[r] * bv[c];
  }
  for (int r = 0; r < R; ++r)
    for (int c = 0; c < C; ++c) {
      double s = acc[r][c][0] + acc[r][c][1];
      if (k < n) s += a[r][k] * b[c][k];
      out[r][c] = s;
    }
}

// The same with four lanes and fused multiply-adds (k mod 4 accumulate apart,
// the lanes are added pairwise at the end, then the last n mod 4 terms).
template <int R, int C>
__attribute__((target("avx2,fma"))) void dots_tile_avx2(const double* const (&a)[R], const double* const (&b)[C],
                                                        int n, double (&out)[R][C]) {
  __m256d acc[R][C];
  for (int r = 0; r < R; ++r)
    for (int c = 0; c < C; ++c) acc[r][c] = _mm256_setzero_pd();
  int k = 0;
  for (; k + 4 <= n; k += 4) {
    __m256d av[R], bv[C];
    for (int r = 0; r < R; ++r) av[r] = _mm256_loadu_pd(a[r] + k);
    for (int c = 0; c < C; ++c) bv[c] = _mm256_loadu_pd(b[c] + k);
    for (int r = 0; r < R; ++r)
      for (int c = 0; c < C; ++c) acc[r][c] = _mm256_fmadd_pd(av[r], bv[c], acc[r][c]);
  }
  for (int r = 0; r < R; ++r)
    for (int c = 0; c < C; ++c) {
      alignas(32) double l[4];
      _mm256_store_pd(l, acc[r][c]);
      double s = (l[0] + l[1]) + (l[2] + l[3]);
      for (int kk = k; kk < n; ++kk) s += a[r][kk] * b[c][kk];
      out[r][c] = s;
    }
}

// Whether the AVX2 form is used: decided once per process from the CPU, so
// every sum of a run is formed the same way whatever the thread count.
inline bool use_avx2() {
  static const bool yes = [] {
    __builtin_cpu_init();
    return __builtin_cpu_supports("avx2") && __builtin_cpu_supports("fma");
  }();
  return yes;
}

template <int R, int C>
inline void dots_tile(const double* const (&a)[R], const double* const (&b)[C], int n, double (&out)[R][C]) {
  if (use_avx2()) dots_tile_avx2<R, C>(a, b, n, out);
  else dots_tile_sse2<R, C>(a, b, n, out);
}

// sum_{k < n} a[k] * b[k] for the short sums (inside a diagonal block, the
// substitutions): always two lanes, inlined.
inline double dot2(const double* a, const double* b, int n) {
  const double* ar[1] = {a};
  const double* br[1] = {b};
  double out[1][1];
  dots_tile_sse2<1, 1>(ar, br, n, out);
  return out[0][0];
}

}  // namespace scoot
