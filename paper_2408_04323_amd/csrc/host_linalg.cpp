// Dense fp64 linear algebra of the host steps (the GP fit and the likelihood
// search, Sec. 4.3): Cholesky factorisation and the inverse of the factor,
// split over the library's host threads with a fixed chunking, so every entry
// is formed by the same sequence of operations whatever the thread count.
#include <algorithm>
#include <cmath>
#include <vector>

#include "host_blas.h"
#include "internal.h"

namespace scoot {

namespace {
constexpr int kChunks = 32;  // work split of every parallel step
constexpr int kBlk = 32;     // block columns of the factorisation
}  // namespace

// Left-looking by block columns of kBlk.  For block columns J .. je-1:
//   1. every row i >= J subtracts from its entries in these columns the
//      products with the factored columns 0 .. J-1 (rows in parallel, tiles of
//      4 rows x 2 columns);
//   2. the diagonal block's rows are factored on the calling thread:
//      (i, j) = (A[i][j] - sum_{J<=k<j} L[i][k] L[j][k]) / L[j][j];
//   3. the rows below form their entries of the block's columns the same way
//      (rows in parallel).
// A pivot that is not positive, or not above 1e-13 of the original diagonal
// entry, means A is not numerically positive definite.
bool cholesky_lower(double* L, int m) {
  std::vector<double> diag(m);
  for (int i = 0; i < m; ++i) diag[i] = L[(size_t)i * m + i];
  for (int J = 0; J < m; J += kBlk) {
    const int je = std::min(m, J + kBlk);
    if (J > 0) {
      const int groups = (m - J + 3) / 4;
      parallel_chunks(kChunks, [&](int c) {
        for (int g = c; g < groups; g += kChunks) {
          const int i0 = J + 4 * g;
          const double* a[4];
          for (int r = 0; r < 4; ++r) a[r] = L + (size_t)std::min(i0 + r, m - 1) * m;
          for (int j0 = J; j0 < je && j0 <= i0 + 3; j0 += 2) {
            const double* b[2] = {L + (size_t)j0 * m, L + (size_t)std::min(j0 + 1, je - 1) * m};
            double s[4][2];
            dots_tile<4, 2>(a, b, J, s);
            for (int r = 0; r < 4; ++r)
              for (int q = 0; q < 2; ++q) {
                const int i = i0 + r, j = j0 + q;
                if (i < m && j < je && j <= i) L[(size_t)i * m + j] -= s[r][q];
              }
          }
        }
      });
    }
    for (int i = J; i < je; ++i) {
      double* Li = L + (size_t)i * m;
      for (int j = J; j <= i; ++j) {
        const double* Lj = L + (size_t)j * m;
        const double s = Li[j] - dot2(Li + J, Lj + J, j - J);
        if (i == j) {
          if (!(s > 1e-13 * diag[i])) return false;
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
          Li[j] = (Li[j] - dot2(Li + J, Lj + J, j - J)) / Lj[j];
        }
      }
    });
  }
  for (int i = 0; i < m; ++i)
    for (int j = i + 1; j < m; ++j) L[(size_t)i * m + j] = 0.0;
  return true;
}

// Columns of L^-1 four at a time (forward substitution of L w = e_j for
// j = j0 .. j0+3, one row of L feeding all four), groups of columns in
// parallel.  Column j is zero above row j; the sums run from row j0, over
// those zeros.
void lower_inverse(const double* L, int m, double* out, bool transposed) {
  const int groups = (m + 3) / 4;
  parallel_chunks(kChunks, [&](int ch) {
    std::vector<double> tmp((size_t)4 * m);
    for (int g = ch; g < groups; g += kChunks) {
      const int j0 = 4 * g, nc = std::min(4, m - j0), top = std::min(m, j0 + 4);
      double* w[4];
      for (int c = 0; c < 4; ++c) w[c] = transposed && c < nc ? out + (size_t)(j0 + c) * m : tmp.data() + (size_t)c * m;
      for (int c = 0; c < 4; ++c)
        for (int i = j0; i < top; ++i) w[c][i] = 0.0;
      for (int i = j0; i < top; ++i) {
        const double* Lr = L + (size_t)i * m;
        for (int c = 0; c < nc; ++c) {
          const int j = j0 + c;
          if (i == j) w[c][i] = 1.0 / Lr[i];
          else if (i > j) w[c][i] = -dot2(Lr + j0, w[c] + j0, i - j0) / Lr[i];
        }
      }
      for (int i = top; i < m; ++i) {
        const double* Lr = L + (size_t)i * m;
        const double* a[1] = {Lr + j0};
        const double* b[4] = {w[0] + j0, w[1] + j0, w[2] + j0, w[3] + j0};
        double s[1][4];
        dots_tile<1, 4>(a, b, i - j0, s);
        for (int c = 0; c < 4; ++c) w[c][i] = -s[0][c] / Lr[i];
      }
      if (!transposed)
        for (int c = 0; c < nc; ++c)
          for (int i = j0 + c; i < m; ++i) out[(size_t)i * m + j0 + c] = w[c][i];
    }
  });
}

}  // namespace scoot
