// Random-forest probability of feasibility and the mask POF(x) >= Delta
// (Sec. 4.7, Eq. 3), on integers: votes = sum over trees of the Q16 value of
// the leaf reached; mask = votes >= ceil(Delta * T * 65536).
//
// The packed trees of one chunk (at most 64 KiB, children adjacent) are
// staged in LDS once per workgroup; each thread owns one candidate, keeps its
// features in its own LDS column (features are indexed dynamically) and walks
// every tree of the chunk, four trees at a time so their dependent LDS reads
// overlap: left iff x[f] <= threshold, a plain float32 compare (NaN goes right).  Forests larger than one chunk take one launch per chunk,
// the vote counts carried in the votes array between launches.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"

namespace scoot {

constexpr int kForestThreads = 512;
constexpr int kWalks = 4;

struct ForestArgs {
  int64_t n;
  int d, n_trees, t_begin, t_end;
  uint32_t node_base, n_nodes;
  int first, last;
  int32_t vote_min;
};

__global__ __launch_bounds__(kForestThreads) void forest_kernel(
    const uint2* __restrict__ nodes, const uint32_t* __restrict__ root, const float* __restrict__ Xc,
    int32_t* __restrict__ votes, uint8_t* __restrict__ mask, int32_t* __restrict__ leaf_idx,
    const ForestArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint2* tree = reinterpret_cast<uint2*>(smem);
  float* xs = reinterpret_cast<float*>(tree + a.n_nodes);  // [d][kForestThreads]
  const int tid = threadIdx.x;
  for (uint32_t i = tid; i < a.n_nodes; i += kForestThreads) tree[i] = nodes[a.node_base + i];
  __syncthreads();

  for (int64_t g = blockIdx.x; g * kForestThreads < a.n; g += gridDim.x) {
    const int64_t c = g * kForestThreads + tid;
    if (c >= a.n) continue;
    for (int k = 0; k < a.d; ++k) xs[k * kForestThreads + tid] = Xc[c * a.d + k];
    int32_t v = a.first ? 0 : votes[c];
    // Four walks in flight, branch-free: all node reads, then all feature
    // reads, then the steps; a finished walk stays on its leaf.
    for (int t0 = a.t_begin; t0 < a.t_end; t0 += kWalks) {
      uint32_t node[kWalks];
      bool live[kWalks];
#pragma unroll
      for (int q = 0; q < kWalks; ++q) {
        live[q] = t0 + q < a.t_end;
        node[q] = live[q] ? root[t0 + q] - a.node_base : root[t0] - a.node_base;
      }
      while (live[0] || live[1] || live[2] || live[3]) {
        uint2 rec[kWalks];
        float x[kWalks];
#pragma unroll
        for (int q = 0; q < kWalks; ++q) rec[q] = tree[node[q]];
#pragma unroll
        for (int q = 0; q < kWalks; ++q) x[q] = xs[(rec[q].x & 31u) * kForestThreads + tid];
#pragma unroll
        for (int q = 0; q < kWalks; ++q) {
          const bool leaf = (rec[q].x & kLeafFlag) != 0;
          if (leaf && live[q]) {
            v += (int32_t)rec[q].y;
            if (leaf_idx) leaf_idx[c * a.n_trees + t0 + q] = (int32_t)(rec[q].x >> 6);
          }
          live[q] = live[q] && !leaf;
          node[q] = leaf ? node[q] : (rec[q].x >> 6) + (x[q] <= __uint_as_float(rec[q].y) ? 0u : 1u);
        }
      }
    }
    if (votes) votes[c] = v;
    if (a.last && mask) mask[c] = v >= a.vote_min ? 1 : 0;
  }
}

int launch_forest(const ForestDevice& f, const float* Xc, int64_t n, int64_t vote_min, int32_t* votes,
                  uint8_t* mask, int32_t* leaf_idx, void* stream) {
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
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)forest_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    attr_set = true;
  }
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
    hipLaunchKernelGGL(forest_kernel, dim3((unsigned)grid), dim3(kForestThreads), lds, s,
                       (const uint2*)f.nodes, f.root, Xc, votes, mask, leaf_idx, a);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("forest launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}

}  // namespace scoot

namespace scoot {

__global__ void fill_u8_kernel(uint8_t* __restrict__ p, int64_t n, uint8_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

int launch_fill_u8(uint8_t* p, int64_t n, uint8_t v, void* stream) {
  if (n == 0) return SCOOT_OK;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(fill_u8_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, p, n, v);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("fill launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}

}  // namespace scoot
