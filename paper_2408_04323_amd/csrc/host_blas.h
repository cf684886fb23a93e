// Register-blocked inner products for the host's dense fp64 steps (Cholesky
// factor, inverse factor, K^-1 in the likelihood gradient).  Every sum has a
// fixed order that depends only on its length (even and odd k accumulate in
// the two lanes of a 16-byte vector, the lanes are added at the end, then an
// odd last term), so results do not depend on how work is split over threads.
#pragma once

#include <cstring>

namespace scoot {

typedef double v2d __attribute__((vector_size(16)));

inline v2d load2(const double* p) {
  v2d v;
  std::memcpy(&v, p, sizeof v);
  return v;
}

// out[r][c] = sum_{k < n} a[r][k] * b[c][k].
template <int R, int C>
inline void dots_tile(const double* const (&a)[R], const double* const (&b)[C], int n, double (&out)[R][C]) {
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

// sum_{k < n} a[k] * b[k], in the same order as dots_tile.
inline double dot2(const double* a, const double* b, int n) {
  const double* ar[1] = {a};
  const double* br[1] = {b};
  double out[1][1];
  dots_tile<1, 1>(ar, br, n, out);
  return out[0][0];
}

}  // namespace scoot
