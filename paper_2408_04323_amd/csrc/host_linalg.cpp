// Dense fp64 linear algebra of the host steps (the GP fit and the likelihood
// search, Sec. 4.3): Cholesky factorisation and the inverse of the factor,
// split over the library's host threads with a fixed chunking, so every entry
// is formed by the same sequence of operations whatever the thread count.
#include <algorithm>
#include <cmath>

#include "internal.h"

namespace scoot {

namespace {
constexpr int kChunks = 32;  // work split of every parallel step
constexpr int kBlk = 32;     // block columns of the factorisation

double dot(const double* a, const double* b, int n) {
  double s = 0.0;
#pragma omp simd reduction(+ : s)
  for (int k = 0; k < n; ++k) s += a[k] * b[k];
  return s;
}
}  // namespace

// Left-looking by block columns of kBlk: the diagonal block's rows are
// factored on the calling thread (the plain row algorithm: entry (i, j) is
// (A[i][j] - sum_{k<j} L[i][k] L[j][k]) / L[j][j]), then every row below the
// block forms its entries of the block's columns the same way, rows in
// parallel (they depend only on the block's rows and on their own earlier
// entries).
bool cholesky_lower(double* L, int m) {
  for (int J = 0; J < m; J += kBlk) {
    const int je = std::min(m, J + kBlk);
    for (int i = J; i < je; ++i) {
      double* Li = L + (size_t)i * m;
      for (int j = J; j <= i; ++j) {
        const double* Lj = L + (size_t)j * m;
        const double s = Li[j] - dot(Li, Lj, j);
        if (i == j) {
          if (!(s > 1e-13 * Li[j])) return false;
          Li[i] = std::sqrt(s);
        } else {
          Li[j] = s / Lj[j];
        }
      }
    }
    if (je == m) break;
    parallel_chunks(kChunks, [&](int c) {
      for (int i = je + c; i < m; i += kChunks) {
        double* Li = L + (size_t)i * m;
        for (int j = J; j < je; ++j) {
          const double* Lj = L + (size_t)j * m;
          Li[j] = (Li[j] - dot(Li, Lj, j)) / Lj[j];
        }
      }
    });
  }
  for (int i = 0; i < m; ++i)
    for (int j = i + 1; j < m; ++j) L[(size_t)i * m + j] = 0.0;
  return true;
}

// Column j of L^-1 by forward substitution of L w = e_j, columns in parallel.
void lower_inverse(const double* L, int m, double* out, bool transposed) {
  parallel_chunks(kChunks, [&](int c) {
    std::vector<double> col;
    if (!transposed) col.resize(m);
    for (int j = c; j < m; j += kChunks) {
      double* w = transposed ? out + (size_t)j * m : col.data();
      w[j] = 1.0 / L[(size_t)j * m + j];
      for (int i = j + 1; i < m; ++i) {
        const double* Lr = L + (size_t)i * m;
        w[i] = -dot(Lr + j, w + j, i - j) / Lr[i];
      }
      if (!transposed)
        for (int i = j; i < m; ++i) out[(size_t)i * m + j] = w[i];
    }
  });
}

}  // namespace scoot
