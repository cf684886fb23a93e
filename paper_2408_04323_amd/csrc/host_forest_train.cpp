// Training the feasibility forest on the host (Sec. 4.7: a random forest
// regressor on every evaluated configuration, label 1 = ran, 0 = crashed).
//
// Every tree is grown by exhaustive search: a node holding samples S with
// bootstrap multiplicities w splits on the feature and threshold maximising
// sum_L^2 / w_L + sum_R^2 / w_R (the decrease of the weighted squared
// deviation of the labels, up to terms that do not depend on the split).  The
// features are rounded to float32 first; thresholds are a/2 + b/2 between
// consecutive distinct values a < b (a if that rounds up to b); equal scores
// go to the lower feature, then the lower threshold.  A node is a leaf (value:
// weighted mean label) at max_depth, with fewer than two distinct samples,
// when its labels are all equal, or when no split beats the unsplit node.
// Tree t draws its bootstrap sample with SplitMix64: draw j picks sample
// floor(u n), u = (output t n + j from `seed`) >> 11 over 2^53.  Nodes are
// numbered in preorder, left child first.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "internal.h"

namespace scoot {

namespace {
uint64_t splitmix64_host(uint64_t seed, uint64_t i) {
  uint64_t z = seed + (i + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

struct Grower {
  const std::vector<double>& X;  // n x d, float32-rounded
  const double* y;
  const std::vector<double>& w;
  int n, d, max_depth;
  TrainedForest& out;
  std::vector<int> order;  // scratch

  int grow(std::vector<int>& idx, int depth) {
    const int me = (int)out.feature.size();
    double W = 0.0, total = 0.0;
    for (int i : idx) {
      W += w[i];
      total += w[i] * y[i];
    }
    out.feature.push_back(-1);
    out.threshold.push_back(0.0);
    out.left.push_back(-1);
    out.right.push_back(-1);
    out.value.push_back(total / W);
    bool pure = true;
    for (int i : idx) pure = pure && y[i] == y[idx[0]];
    if (depth >= max_depth || idx.size() < 2 || pure) return me;

    double best = total * total / W;  // a split must beat the unsplit node
    int best_f = -1;
    double best_t = 0.0;
    for (int f = 0; f < d; ++f) {
      order = idx;
      std::stable_sort(order.begin(), order.end(),
                       [&](int a, int b) { return X[(size_t)a * d + f] < X[(size_t)b * d + f]; });
      double sl = 0.0, wl = 0.0;
      for (size_t p = 0; p + 1 < order.size(); ++p) {
        sl += w[order[p]] * y[order[p]];
        wl += w[order[p]];
        const double xa = X[(size_t)order[p] * d + f], xb = X[(size_t)order[p + 1] * d + f];
        if (xb == xa) continue;
        const double sr = total - sl, wr = W - wl;
        const double proxy = sl * sl / wl + sr * sr / wr;
        if (proxy > best) {
          best = proxy;
          best_f = f;
          const double t = xa / 2.0 + xb / 2.0;
          best_t = t == xb ? xa : t;
        }
      }
    }
    if (best_f < 0) return me;
    std::vector<int> li, ri;
    for (int i : idx) (X[(size_t)i * d + best_f] <= best_t ? li : ri).push_back(i);
    out.feature[me] = best_f;
    out.threshold[me] = best_t;
    const int l = grow(li, depth + 1);
    out.left[me] = l;
    const int r = grow(ri, depth + 1);
    out.right[me] = r;
    return me;
  }
};
}  // namespace

int train_forest_host(const double* X, const double* y, int n, int d, int n_trees, int max_depth, uint64_t seed,
                      bool bootstrap, TrainedForest& out) {
  if (!X || !y) return fail(SCOOT_ERR_INVALID_ARG, "forest train: null pointer");
  if (n < 1 || d < 1 || n_trees < 1 || max_depth < 0)
    return fail(SCOOT_ERR_INVALID_ARG, "forest train: bad n, d, n_trees or max_depth");
  if (d > SCOOT_MAX_DIM) return fail(SCOOT_ERR_UNSUPPORTED, "forest train: d exceeds SCOOT_MAX_DIM");
  if (n_trees > SCOOT_MAX_TREES) return fail(SCOOT_ERR_UNSUPPORTED, "forest train: too many trees");
  if (max_depth > 64) return fail(SCOOT_ERR_UNSUPPORTED, "forest train: max_depth above 64");
  std::vector<double> X32((size_t)n * d);
  for (size_t i = 0; i < (size_t)n * d; ++i) {
    if (!std::isfinite(X[i])) return fail(SCOOT_ERR_INVALID_ARG, "forest train: non-finite input");
    X32[i] = (double)(float)X[i];
  }
  for (int i = 0; i < n; ++i)
    if (!std::isfinite(y[i])) return fail(SCOOT_ERR_INVALID_ARG, "forest train: non-finite label");
  // Trees are independent: each is grown on its own (tree t by chunk
  // t mod the chunk count) and the forest is put together in tree order.
  std::vector<TrainedForest> trees(n_trees);
  const int n_chunks = std::min(n_trees, 64);
  parallel_chunks(n_chunks, [&](int c) {
    std::vector<double> w(n);
    for (int t = c; t < n_trees; t += n_chunks) {
      if (bootstrap) {
        std::fill(w.begin(), w.end(), 0.0);
        for (int j = 0; j < n; ++j) {
          const uint64_t r = splitmix64_host(seed, (uint64_t)t * (uint64_t)n + (uint64_t)j);
          const double u = (double)(r >> 11) * (1.0 / 9007199254740992.0);
          w[(int)(u * n)] += 1.0;
        }
      } else {
        std::fill(w.begin(), w.end(), 1.0);
      }
      std::vector<int> idx;
      for (int i = 0; i < n; ++i)
        if (w[i] > 0) idx.push_back(i);
      Grower g{X32, y, w, n, d, max_depth, trees[t], {}};
      g.grow(idx, 0);  // node indices come out tree-local
    }
  });
  out = TrainedForest();
  out.tree_offset.push_back(0);
  for (int t = 0; t < n_trees; ++t) {
    const TrainedForest& tr = trees[t];
    if (tr.feature.size() > (size_t)kChunkNodes - 1)
      return fail(SCOOT_ERR_UNSUPPORTED, "forest train: a tree has more than 8191 nodes (lower max_depth)");
    out.feature.insert(out.feature.end(), tr.feature.begin(), tr.feature.end());
    out.threshold.insert(out.threshold.end(), tr.threshold.begin(), tr.threshold.end());
    out.left.insert(out.left.end(), tr.left.begin(), tr.left.end());
    out.right.insert(out.right.end(), tr.right.begin(), tr.right.end());
    out.value.insert(out.value.end(), tr.value.begin(), tr.value.end());
    out.tree_offset.push_back((int64_t)out.feature.size());
  }
  return SCOOT_OK;
}

}  // namespace scoot
