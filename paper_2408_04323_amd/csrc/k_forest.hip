// Random-forest probability of feasibility and the mask POF(x) >= Delta
// (Sec. 4.7, Eq. 3), on integers: votes = sum over trees of the Q16 value of
// the leaf reached; mask = votes >= ceil(Delta * T * 65536).
//
// The packed trees of one chunk (at most 64 KiB, children adjacent) are
// staged in LDS once per workgroup; each thread owns one candidate, keeps its
// features in its own LDS column (features are indexed dynamically) and walks
// four trees at a time.  A step is branch-free: read the node, read the
// feature it names, go to child + (x <= threshold ? 0 : 1) (a float32
// compare; NaN goes right).  Leaves carry a NaN threshold and point one below
// themselves, so a walk that has arrived stays put; each group of trees runs
// exactly as many steps as its deepest tree (the host orders the trees deepest
// first, so the four are alike), then reads the leaves' values from the NaN
// payloads.  Forests larger than one chunk take one launch per
// chunk, the vote counts carried in the votes array between launches.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"

namespace scoot {

constexpr int kForestThreads = kForestThreadsPerBlock;
constexpr int kWalks = 4;
static_assert(kForestThreads * 4 == (1 << 11), "feature << 11 is the byte offset of a feature column");

typedef __attribute__((address_space(3))) const float lds_f32;  // an LDS address

struct ForestArgs {
  int64_t n;
  int d, n_trees, t_begin, t_end;
  uint32_t node_base, n_nodes;
  int first, last;
  int32_t vote_min;
};

__global__ __launch_bounds__(kForestThreads) void forest_kernel(
    const uint2* __restrict__ nodes, const uint32_t* __restrict__ root, const uint32_t* __restrict__ depth,
    const int32_t* __restrict__ leaf_orig, const int32_t* __restrict__ tree_orig, const float* __restrict__ Xc,
    int32_t* __restrict__ votes,
    uint8_t* __restrict__ mask, int32_t* __restrict__ leaf_idx, const uint8_t* __restrict__ known,
    const ForestArgs a) {
  // LDS: the feature columns [d][kForestThreads] floats at LDS address 0 (the
  // kernel declares no static LDS, so its dynamic LDS starts there), so that a
  // thread's feature address is (feature << 11) | (tid * 4), one and-or; then
  // the chunk's nodes.
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* xs = smem;
  uint2* tree = reinterpret_cast<uint2*>(smem + (size_t)a.d * kForestThreads * 4);
  const int tid = threadIdx.x;
  for (uint32_t i = tid; i < a.n_nodes; i += kForestThreads) tree[i] = nodes[a.node_base + i];
  __syncthreads();
  const uint32_t lane4 = (uint32_t)tid * 4u;
  for (int64_t g = blockIdx.x; g * kForestThreads < a.n; g += gridDim.x) {
    const int64_t c = g * kForestThreads + tid;
    if (c >= a.n) continue;
    for (int k = 0; k < a.d; ++k) reinterpret_cast<float*>(xs)[k * kForestThreads + tid] = Xc[c * a.d + k];
    int32_t v = a.first ? 0 : votes[c];
    for (int t0 = a.t_begin; t0 < a.t_end; t0 += kWalks) {
      const int cnt = min(kWalks, a.t_end - t0);
      uint32_t node[kWalks];
      uint32_t steps = 0;
#pragma unroll
      for (int q = 0; q < kWalks; ++q) {
        const int t = q < cnt ? t0 + q : t0;
        node[q] = root[t] - a.node_base;
        steps = max(steps, depth[t]);
      }
      steps = __builtin_amdgcn_readfirstlane(steps);  // the same for every lane: a scalar loop count
      for (uint32_t s = 0; s < steps; ++s) {
        uint2 rec[kWalks];
        float x[kWalks];
#pragma unroll
        for (int q = 0; q < kWalks; ++q) rec[q] = tree[node[q]];
#pragma unroll
        for (int q = 0; q < kWalks; ++q) x[q] = *reinterpret_cast<const lds_f32*>((size_t)((rec[q].x & 0x7800u) | lane4));
#pragma unroll
        for (int q = 0; q < kWalks; ++q) node[q] = (rec[q].x >> 15) + (x[q] <= __uint_as_float(rec[q].y) ? 0u : 1u);
      }
#pragma unroll
      for (int q = 0; q < kWalks; ++q) {
        if (q < cnt) {
          v += (int32_t)(tree[node[q]].y & 0x1FFFFu);
          if (leaf_idx) leaf_idx[c * a.n_trees + tree_orig[t0 + q]] = leaf_orig[a.node_base + node[q]];
        }
      }
    }
    if (votes) votes[c] = v;
    if (a.last && mask) mask[c] = v >= a.vote_min && (!known || known[c] != 0) ? 1 : 0;
  }
}

int launch_forest(const ForestDevice& f, const float* Xc, int64_t n, int64_t vote_min, int32_t* votes,
                  uint8_t* mask, int32_t* leaf_idx, void* stream, const uint8_t* known) {
  if (n == 0) return SCOOT_OK;
  hipStream_t s = (hipStream_t)stream;
  const int n_chunks = (int)f.chunk_tree.size() - 1;
  if (n_chunks > 1 && !votes) {
    votes = (int32_t*)device_scratch((size_t)n * 4, 2);
    if (!votes) return fail(SCOOT_ERR_NO_MEMORY, "forest: vote scratch allocation failed");
  }
  int dev = 0, cus = 256;
  (void)hipGetDevice(&dev);
  (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  // As many workgroups as the LDS of a CU holds (each stages the largest chunk).
  uint32_t max_nodes = 0;
  for (int ch = 0; ch < n_chunks; ++ch)
    max_nodes = std::max(max_nodes, f.chunk_first_node[ch + 1] - f.chunk_first_node[ch]);
  const size_t lds_max = (size_t)max_nodes * 8 + (size_t)f.d * kForestThreads * 4;
  const int per_cu = std::max(1, std::min(4, (int)((160 * 1024) / lds_max)));
  int64_t groups = (n + kForestThreads - 1) / kForestThreads;
  int64_t grid = std::min(groups, (int64_t)cus * per_cu);
  const int rc = allow_full_lds((const void*)forest_kernel, "forest");
  if (rc != SCOOT_OK) return rc;
  for (int ch = 0; ch < n_chunks; ++ch) {
    ForestArgs a{};
    a.n = n;
    a.d = f.d;
    a.n_trees = f.n_trees;
    a.t_begin = f.chunk_tree[ch];
    a.t_end = f.chunk_tree[ch + 1];
    a.node_base = f.chunk_first_node[ch];
    a.n_nodes = f.chunk_first_node[ch + 1] - f.chunk_first_node[ch];
    a.first = ch == 0;
    a.last = ch == n_chunks - 1;
    a.vote_min = (int32_t)vote_min;
    const size_t lds = (size_t)a.n_nodes * 8 + (size_t)f.d * kForestThreads * 4;
    hipLaunchKernelGGL(forest_kernel, dim3((unsigned)grid), dim3(kForestThreads), lds, s, (const uint2*)f.nodes,
                       f.root, f.depth, f.leaf_orig, f.tree_orig, Xc, votes, mask, leaf_idx, known, a);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("forest launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}

}  // namespace scoot
