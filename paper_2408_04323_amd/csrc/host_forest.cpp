// Host side of the random-forest feasibility mask (Sec. 4.7, Eq. 3): checks
// the flat tree arrays and repacks every tree breadth-first so that the two
// children of a node are adjacent (one child index per node), 8 bytes per
// node (encoding in internal.h), orders the trees deepest first (a thread
// walks four trees for as many steps as the deepest of them; votes are sums,
// so the order does not change them) and groups consecutive trees into chunks
// that fit the on-chip memory of one workgroup.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <deque>

#include "internal.h"

namespace scoot {

int pack_forest(const int32_t* feature, const float* threshold, const int32_t* left,
                const int32_t* right, const int32_t* leaf_q16, const int64_t* tree_offset,
                int n_trees, int d, ForestHost& fh) {
  if (!feature || !threshold || !left || !right || !leaf_q16 || !tree_offset)
    return fail(SCOOT_ERR_INVALID_ARG, "forest: null pointer");
  if (n_trees < 1 || n_trees > SCOOT_MAX_TREES) return fail(SCOOT_ERR_INVALID_ARG, "forest: bad tree count");
  if (d < 1 || d > SCOOT_MAX_DIM) return fail(SCOOT_ERR_INVALID_ARG, "forest: bad d");
  if (tree_offset[0] != 0) return fail(SCOOT_ERR_INVALID_ARG, "forest: tree_offset[0] must be 0");
  fh = ForestHost();
  fh.n_trees = n_trees;
  fh.d = d;

  // Breadth-first order of each tree, validated, with its depth.
  std::vector<std::vector<int>> order(n_trees);
  fh.depth.assign(n_trees, 0);
  for (int t = 0; t < n_trees; ++t) {
    int64_t base = tree_offset[t], size = tree_offset[t + 1] - base;
    if (size < 1 || size > kChunkNodes - 1)
      return fail(size < 1 ? SCOOT_ERR_INVALID_ARG : SCOOT_ERR_UNSUPPORTED,
                  "forest: empty tree or tree larger than 8191 nodes");
    std::vector<int> level(size, -1);
    std::deque<int> q{0};
    level[0] = 0;
    while (!q.empty()) {
      int u = q.front();
      q.pop_front();
      order[t].push_back(u);
      fh.depth[t] = std::max<uint32_t>(fh.depth[t], (uint32_t)level[u]);
      int64_t g = base + u;
      int L = left[g], R = right[g];
      if (L < 0 && R < 0) {
        if (leaf_q16[g] < 0 || leaf_q16[g] > 65536)
          return fail(SCOOT_ERR_INVALID_ARG, "forest: leaf value outside [0, 65536]");
        continue;
      }
      if (L < 0 || R < 0 || L >= size || R >= size || L == R)
        return fail(SCOOT_ERR_INVALID_ARG, "forest: bad child index");
      if (feature[g] < 0 || feature[g] >= d) return fail(SCOOT_ERR_INVALID_ARG, "forest: bad feature index");
      if (std::isnan(threshold[g])) return fail(SCOOT_ERR_INVALID_ARG, "forest: NaN threshold");
      for (int c : {L, R}) {
        if (level[c] >= 0) return fail(SCOOT_ERR_INVALID_ARG, "forest: node reached twice (not a tree)");
        level[c] = level[u] + 1;
        q.push_back(c);
      }
    }
  }

  // Slots: trees deepest first, ties by index.
  fh.tree_orig.resize(n_trees);
  for (int t = 0; t < n_trees; ++t) fh.tree_orig[t] = t;
  std::stable_sort(fh.tree_orig.begin(), fh.tree_orig.end(),
                   [&](int a, int b) { return fh.depth[a] > fh.depth[b]; });
  {
    std::vector<uint32_t> by_slot(n_trees);
    for (int s = 0; s < n_trees; ++s) by_slot[s] = fh.depth[fh.tree_orig[s]];
    fh.depth = by_slot;
  }

  // Chunks of consecutive slots: one unused node, then whole trees, at most
  // kChunkNodes nodes in all.
  fh.chunk_tree.push_back(0);
  int in_chunk = 1;
  for (int s = 0; s < n_trees; ++s) {
    const int t = fh.tree_orig[s];
    int sz = (int)order[t].size();
    if (in_chunk + sz > kChunkNodes) {
      fh.chunk_tree.push_back(s);
      in_chunk = 1;
    }
    in_chunk += sz;
  }
  fh.chunk_tree.push_back(n_trees);

  // Pack.  Child indices are relative to the chunk's first (unused) node.
  size_t total = (fh.chunk_tree.size() - 1);
  for (auto& o : order) total += o.size();
  fh.nodes.assign(total * 2, 0);
  fh.leaf_orig.assign(total, -1);
  fh.root.assign(n_trees + 1, 0);
  uint32_t next = 0;
  for (size_t ch = 0; ch + 1 < fh.chunk_tree.size(); ++ch) {
    const uint32_t chunk_first = next;
    fh.chunk_first_node.push_back(chunk_first);
    fh.nodes[2 * next] = 0;  // the unused node
    fh.nodes[2 * next + 1] = kLeafNaN;
    ++next;
    for (int s = fh.chunk_tree[ch]; s < fh.chunk_tree[ch + 1]; ++s) {
      const int t = fh.tree_orig[s];
      int64_t base = tree_offset[t];
      std::vector<uint32_t> pos(tree_offset[t + 1] - base, 0);
      uint32_t cursor = next;
      pos[0] = cursor++;
      for (int u : order[t]) {
        int64_t g = base + u;
        if (left[g] >= 0) {
          pos[left[g]] = cursor++;
          pos[right[g]] = cursor++;
        }
      }
      fh.root[s] = pos[0];
      for (int u : order[t]) {
        int64_t g = base + u;
        uint32_t at = pos[u];
        uint32_t rel = at - chunk_first;
        if (left[g] < 0) {
          fh.nodes[2 * at] = (rel - 1) << 15;
          fh.nodes[2 * at + 1] = kLeafNaN | (uint32_t)leaf_q16[g];
          fh.leaf_orig[at] = u;
        } else {
          uint32_t child = pos[left[g]] - chunk_first;
          fh.nodes[2 * at] = (child << 15) | ((uint32_t)feature[g] << 11);
          uint32_t bits;
          std::memcpy(&bits, &threshold[g], 4);
          fh.nodes[2 * at + 1] = bits;
        }
      }
      next = cursor;
    }
  }
  fh.root[n_trees] = next;
  fh.chunk_first_node.push_back(next);
  return SCOOT_OK;
}

}  // namespace scoot
