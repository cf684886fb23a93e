// Host side of EHVI (Sec. 4.4.2, Eq. 9): the Pareto front of the observed
// values and a partition into boxes of the region below the reference point
// that the front leaves open (objectives minimised, r an upper bound).
//
// With G_j(c) = E[(c - Y_j)^+] the improvement of one box B = [l, u] has
// expectation prod_j (G_j(u_j) - G_j(l_j)), so the device only needs, per
// axis, the distinct box coordinates and, per box, index pairs into them.
//
// Boxes: the sorted front coordinates (with -inf and r) grid the first p-1
// axes; over each grid cell the open region is [-inf, h] along the last axis,
// h = min(r, last coordinate of the front points that dominate the cell's
// lower corner).  For three objectives, consecutive cells along the second
// axis with the same h are merged into one box.
#include <algorithm>
#include <cmath>
#include <limits>

#include "internal.h"

namespace scoot {

int build_boxes(const double* Y, int m, int p, const double* ref, BoxTable& bt) {
  if (p < 1 || p > SCOOT_MAX_OBJECTIVES) return fail(SCOOT_ERR_INVALID_ARG, "ehvi: p must be 1..3");
  if (m < 0 || (m > 0 && !Y) || !ref) return fail(SCOOT_ERR_INVALID_ARG, "ehvi: null pointer or m < 0");
  for (int j = 0; j < p; ++j)
    if (!std::isfinite(ref[j])) return fail(SCOOT_ERR_INVALID_ARG, "ehvi: non-finite reference point");
  for (long i = 0; i < (long)m * p; ++i)
    if (!std::isfinite(Y[i])) return fail(SCOOT_ERR_INVALID_ARG, "ehvi: non-finite observed value");

  // Rows strictly below r, sorted lexicographically, duplicates once.
  std::vector<std::vector<double>> rows;
  for (int i = 0; i < m; ++i) {
    bool below = true;
    for (int j = 0; j < p; ++j) below = below && (Y[(size_t)i * p + j] < ref[j]);
    if (below) rows.emplace_back(Y + (size_t)i * p, Y + (size_t)i * p + p);
  }
  std::sort(rows.begin(), rows.end());
  rows.erase(std::unique(rows.begin(), rows.end()), rows.end());
  // Drop rows weakly dominated by another (distinct) row.
  std::vector<std::vector<double>> front;
  for (size_t a = 0; a < rows.size(); ++a) {
    bool dominated = false;
    for (size_t b = 0; b < rows.size() && !dominated; ++b) {
      if (a == b) continue;
      bool le = true, lt = false;
      for (int j = 0; j < p; ++j) {
        le = le && rows[b][j] <= rows[a][j];
        lt = lt || rows[b][j] < rows[a][j];
      }
      dominated = le && lt;
    }
    if (!dominated) front.push_back(rows[a]);
  }

  bt = BoxTable();
  bt.p = p;
  bt.n_front = (int)front.size();
  for (auto& r : front) bt.front.insert(bt.front.end(), r.begin(), r.end());
  const double ninf = -std::numeric_limits<double>::infinity();
  bt.coord.assign(p, {});
  for (int j = 0; j < p; ++j) {
    std::vector<double> v;
    for (auto& r : front) v.push_back(r[j]);
    std::sort(v.begin(), v.end());
    v.erase(std::unique(v.begin(), v.end()), v.end());
    bt.coord[j].push_back(ninf);
    bt.coord[j].insert(bt.coord[j].end(), v.begin(), v.end());
    bt.coord[j].push_back(ref[j]);
    if (bt.coord[j].size() > 32000) return fail(SCOOT_ERR_UNSUPPORTED, "ehvi: front too large");
  }
  auto index_of = [&](int j, double v) {
    const auto& c = bt.coord[j];
    return (int16_t)(std::lower_bound(c.begin() + 1, c.end(), v) - c.begin());
  };
  auto push = [&](const int* lo, const int* hi) {
    for (int j = 0; j < p; ++j) {
      bt.lo.push_back((int16_t)lo[j]);
      bt.hi.push_back((int16_t)hi[j]);
    }
  };
  const int last = p - 1;
  if (p == 1) {
    int lo[1] = {0}, hi[1] = {1};  // (-inf, min front) or (-inf, r)
    push(lo, hi);
    return SCOOT_OK;
  }
  const auto& a = bt.coord[0];
  if (p == 2) {
    for (size_t i = 0; i + 1 < a.size(); ++i) {
      double h = ref[last];
      for (auto& r : front)
        if (r[0] <= a[i]) h = std::min(h, r[last]);
      int lo[2] = {(int)i, 0}, hi[2] = {(int)i + 1, index_of(last, h)};
      push(lo, hi);
    }
    return SCOOT_OK;
  }
  const auto& b = bt.coord[1];
  for (size_t i = 0; i + 1 < a.size(); ++i) {
    size_t j = 0;
    while (j + 1 < b.size()) {
      auto height = [&](size_t jj) {
        double h = ref[last];
        for (auto& r : front)
          if (r[0] <= a[i] && r[1] <= b[jj]) h = std::min(h, r[last]);
        return h;
      };
      double h = height(j);
      size_t k = j + 1;
      while (k + 1 < b.size() && height(k) == h) ++k;
      int lo[3] = {(int)i, (int)j, 0}, hi[3] = {(int)i + 1, (int)k, index_of(last, h)};
      push(lo, hi);
      j = k;
    }
  }
  return SCOOT_OK;
}

}  // namespace scoot
