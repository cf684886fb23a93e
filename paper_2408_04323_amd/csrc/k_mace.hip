// MACE for one objective (Sec. 4.5.1; scores Eq. 6-8), objective minimised:
//
//   ucb = beta * sd - mu               Eq. 6 for -Y (the paper maximises f = -y)
//   pi  = Phi((best + xi - mu) / sd)   Eq. 7: P(Y < best + xi); 1 or 0 when sd = 0
//   ei  = G(best + xi)                 Eq. 8 (normal.h)
//
// then the Pareto front of (ucb, pi, ei) over the eligible candidates, all
// three maximised: a candidate is dominated when another eligible one scores
// at least as high on all three and higher on one.  The random pick from the
// front is in k_select.hip.
//
// Front, by filters that only ever remove dominated candidates (so the result
// is exact: domination is transitive on a finite set, whatever is dominated is
// dominated by a front member, and no front member is ever removed):
//  A. pivots: per tile of 1024 candidates, the maximisers of 13 positive
//     weightings of the tile's range-normalised scores -- strong, spread
//     points (a point that maximises a positive weighting has no dominator,
//     up to rounding; nothing below relies on it);
//  B. the front of the pivot set: every pivot against every pivot, then its
//     members gathered once into a packed list (one global atomic per wave);
//  C. every candidate checked against that list (staged through LDS);
//     survivors set their flag and append their index to a list (one global
//     atomic per wave);
//  D. every listed candidate against every listed one.
// B and D spread (256 owners) x (chunk of 256 in LDS) pairs over a persistent
// grid; a dominated owner clears its flag (several workgroups may clear one
// flag: they all write 0).  The flags do not depend on the order of the list.
// When the three scores agree (the usual case) the pivot front is close to
// the true front and C leaves few candidates for D; in full conflict C and D
// grow to n^2.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "internal.h"
#include "normal.h"

namespace scoot {

constexpr int kMaceThreads = 256;
constexpr int kParetoTile = 1024;   // candidates per stage-1 workgroup, 4 per thread

template <typename T>
__global__ __launch_bounds__(kMaceThreads) void mace_scores_kernel(const T* __restrict__ mu, const T* __restrict__ sd,
                                                                   int64_t n, T c, T beta, T* __restrict__ ucb,
                                                                   T* __restrict__ pi, T* __restrict__ ei) {
  for (int64_t i = (int64_t)blockIdx.x * kMaceThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kMaceThreads) {
    const T m = mu[i], s = sd[i], r = reciprocal(s);
    ucb[i] = beta * s - m;
    pi[i] = s > T(0) ? normal_cdf((c - m) * r) : (m < c ? T(1) : T(0));
    ei[i] = partial_expectation<T>(c, m, s, r);
  }
}

// j dominates i (all >=, one >); false whenever a NaN is involved.
template <typename T>
__device__ inline bool dominates(T ja, T jb, T jc, T ia, T ib, T ic) {
  return ja >= ia && jb >= ib && jc >= ic && (ja > ia || jb > ib || jc > ic);
}

// ---- A: pivots ----------------------------------------------------------------
// Weights (w0, w1, w2) of the tile-normalised scores: the ten with w_k >= 1,
// sum 6, and three near the axes.
constexpr int kPivotsPerTile = 13;
constexpr float kPivotW[kPivotsPerTile][3] = {  // folds into the code as immediates
    {1, 1, 4}, {1, 2, 3}, {1, 3, 2}, {1, 4, 1}, {2, 1, 3}, {2, 2, 2}, {2, 3, 1}, {3, 1, 2}, {3, 2, 1}, {4, 1, 1},
    {16, 1, 1}, {1, 16, 1}, {1, 1, 16}};

// Order-preserving key of (value, local index): larger value first, then the
// lower index; 0 = no candidate.
__device__ inline uint64_t pivot_key(float v, int idx) {
  uint32_t u = __float_as_uint(v + 0.0f);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)idx);
}

template <typename T>
__global__ __launch_bounds__(kMaceThreads) void pareto_pivot_kernel(const T* __restrict__ a, const T* __restrict__ b,
                                                                    const T* __restrict__ c,
                                                                    const uint8_t* __restrict__ mask, int64_t n,
                                                                    T* __restrict__ pa, T* __restrict__ pb,
                                                                    T* __restrict__ pc, uint8_t* __restrict__ pfront,
                                                                    int32_t* __restrict__ count) {
  __shared__ float red[6][kMaceThreads / 64];
  __shared__ uint64_t wave_best[kPivotsPerTile][kMaceThreads / 64];
  __shared__ int piv_idx[kPivotsPerTile];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t base = (int64_t)blockIdx.x * kParetoTile;
  if (blockIdx.x == 0 && tid < 2) count[tid] = 0;  // for the gather and stage C, which run after this kernel
  T v[4][3];
  bool ok[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t i = base + r * kMaceThreads + tid;
    ok[r] = false;
    v[r][0] = v[r][1] = v[r][2] = T(0);
    if (i < n) {
      v[r][0] = a[i];
      v[r][1] = b[i];
      v[r][2] = c[i];
      ok[r] = (!mask || mask[i] != 0) && v[r][0] == v[r][0] && v[r][1] == v[r][1] && v[r][2] == v[r][2];
    }
  }
  // tile range of each score over the eligible candidates (in float: it only
  // shapes the weights), six maxima in one reduction
  float m6[6];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    m6[k] = -INFINITY;
    m6[3 + k] = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      m6[k] = fmaxf(m6[k], ok[r] ? (float)v[r][k] : -INFINITY);
      m6[3 + k] = fmaxf(m6[3 + k], ok[r] ? -(float)v[r][k] : -INFINITY);
    }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1)
#pragma unroll
    for (int k = 0; k < 6; ++k) m6[k] = fmaxf(m6[k], __shfl_xor(m6[k], m));
  if (lane == 0)
#pragma unroll
    for (int k = 0; k < 6; ++k) red[k][wave] = m6[k];
  __syncthreads();
  float lo[3], scale[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    float hi = red[k][0], nlo = red[3 + k][0];
#pragma unroll
    for (int w = 1; w < kMaceThreads / 64; ++w) {
      hi = fmaxf(hi, red[k][w]);
      nlo = fmaxf(nlo, red[3 + k][w]);
    }
    lo[k] = -nlo;
    scale[k] = hi > lo[k] ? 1.0f / (hi - lo[k]) : 0.0f;
  }
  // the 13 weighted maximisers
  // (branch-free: an ineligible candidate's key is 0, which never wins)
  float x[4][3];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int k = 0; k < 3; ++k) x[r][k] = ((float)v[r][k] - lo[k]) * scale[k];
  uint64_t best[kPivotsPerTile];
#pragma unroll
  for (int d = 0; d < kPivotsPerTile; ++d) {
    best[d] = 0;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float val = kPivotW[d][0] * x[r][0] + kPivotW[d][1] * x[r][1] + kPivotW[d][2] * x[r][2];
      const uint64_t key = ok[r] ? pivot_key(val, r * kMaceThreads + tid) : 0;
      best[d] = key > best[d] ? key : best[d];
    }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1)
#pragma unroll
    for (int d = 0; d < kPivotsPerTile; ++d) {
      const uint64_t o = (uint64_t)__shfl_xor((unsigned long long)best[d], m);
      best[d] = o > best[d] ? o : best[d];
    }
  if (lane == 0)
#pragma unroll
    for (int d = 0; d < kPivotsPerTile; ++d) wave_best[d][wave] = best[d];
  __syncthreads();
  if (tid < kPivotsPerTile) {
    uint64_t k = wave_best[tid][0];
    for (int w = 1; w < kMaceThreads / 64; ++w) k = wave_best[tid][w] > k ? wave_best[tid][w] : k;
    piv_idx[tid] = k ? (int)(0xFFFFFFFFu - (uint32_t)k) : -1;
  }
  __syncthreads();
  if (tid < kPivotsPerTile) {
    const int li = piv_idx[tid];
    bool keep = li >= 0;
    for (int k2 = 0; k2 < tid; ++k2) keep = keep && piv_idx[k2] != li;  // each point once
    const int64_t out = (int64_t)blockIdx.x * kPivotsPerTile + tid;
    const int64_t gi = base + (li >= 0 ? li : 0);
    pfront[out] = keep ? 1 : 0;
    pa[out] = keep ? a[gi] : T(0);
    pb[out] = keep ? b[gi] : T(0);
    pc[out] = keep ? c[gi] : T(0);
  }
}

template <typename T>
struct Vec4;
template <>
struct Vec4<float> {
  typedef float type __attribute__((ext_vector_type(4)));
};
template <>
struct Vec4<double> {
  typedef double type __attribute__((ext_vector_type(4)));
};

// ---- B': the pivot front, packed ----------------------------------------------
// Slots whose flag B left set go to front[0 .. count[1]) as (a, b, c, -), in
// no particular order (C only asks whether some member dominates a candidate).
template <typename T>
__global__ __launch_bounds__(kMaceThreads) void pareto_gather_kernel(const T* __restrict__ pa,
                                                                     const T* __restrict__ pb,
                                                                     const T* __restrict__ pc,
                                                                     const uint8_t* __restrict__ pfront, int64_t P,
                                                                     typename Vec4<T>::type* __restrict__ front,
                                                                     int32_t* __restrict__ count) {
  const int lane = threadIdx.x & 63;
  const int64_t k = (int64_t)blockIdx.x * kMaceThreads + threadIdx.x;
  const bool live = k < P && pfront[k] != 0;
  const uint64_t bal = __ballot(live);
  if (!bal) return;
  int at = 0;
  if (lane == 0) at = atomicAdd(count + 1, (int)__popcll(bal));
  at = __shfl(at, 0);
  const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
  if (live) front[at + below] = typename Vec4<T>::type{pa[k], pb[k], pc[k], T(0)};
}

// ---- C: candidates against the pivot front ----------------------------------------
template <typename T>
__global__ __launch_bounds__(kMaceThreads) void pareto_filter_kernel(
    const T* __restrict__ a, const T* __restrict__ b, const T* __restrict__ c, const uint8_t* __restrict__ mask,
    int64_t n, const typename Vec4<T>::type* __restrict__ front, uint8_t* __restrict__ flags,
    int32_t* __restrict__ list, int32_t* __restrict__ count) {
  typedef typename Vec4<T>::type V;
  __shared__ V pts[kParetoTile];
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t base = (int64_t)blockIdx.x * kParetoTile;
  const int64_t F = count[1];  // size of the packed pivot front
  T va[4], vb[4], vc[4];
  bool alive[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t i = base + r * kMaceThreads + tid;
    alive[r] = false;
    va[r] = vb[r] = vc[r] = T(0);
    if (i < n) {
      va[r] = a[i];
      vb[r] = b[i];
      vc[r] = c[i];
      alive[r] = (!mask || mask[i] != 0) && va[r] == va[r] && vb[r] == vb[r] && vc[r] == vc[r];
    }
  }
  for (int64_t cb = 0; cb < F; cb += kParetoTile) {
    const int live = (int)std::min<int64_t>(kParetoTile, F - cb);
    __syncthreads();  // the previous chunk is no longer read
    for (int k = tid; k < live; k += kMaceThreads) pts[k] = front[cb + k];
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (alive[r])
        for (int j = 0; j < live; ++j)
          if (dominates(pts[j].x, pts[j].y, pts[j].z, va[r], vb[r], vc[r])) {
            alive[r] = false;
            break;
          }
    if (!__syncthreads_or(alive[0] || alive[1] || alive[2] || alive[3])) break;
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t i = base + r * kMaceThreads + tid;
    if (i < n) flags[i] = alive[r] ? 1 : 0;
    const uint64_t bal = __ballot(alive[r]);
    if (bal) {
      int at = 0;
      if (lane == 0) at = atomicAdd(count, (int)__popcll(bal));
      at = __shfl(at, 0);
      const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
      if (alive[r]) list[at + below] = (int32_t)i;
    }
  }
}

constexpr int kMergeChunk = 256;

// B and D.  Owners and dominators are the S entries of `list` (S = *count),
// or, when list is null, the slots 0..S_slots-1 themselves with flags[]
// telling which hold a point (an empty slot neither owns nor dominates).
// Each (256 owners) x (chunk of 256) item stages the chunk's points, packed
// (a, b, c, -) and compacted, in LDS; owners test four at a time.
template <typename T>
__global__ __launch_bounds__(kMaceThreads) void pareto_merge_kernel(const T* __restrict__ a, const T* __restrict__ b,
                                                                    const T* __restrict__ c,
                                                                    const int32_t* __restrict__ list,
                                                                    const int32_t* __restrict__ count, int64_t S_slots,
                                                                    uint8_t* __restrict__ flags) {
  typedef typename Vec4<T>::type V;
  __shared__ V pts[kMergeChunk];
  __shared__ int n_live;
  const int tid = threadIdx.x;
  const int64_t S = list ? (int64_t)*count : S_slots;
  const int64_t nb = (S + kMaceThreads - 1) / kMaceThreads, nc = (S + kMergeChunk - 1) / kMergeChunk;
  for (int64_t item = blockIdx.x; item < nb * nc; item += gridDim.x) {
    const int64_t s = (item / nc) * kMaceThreads + tid;
    const int64_t cb = (item % nc) * kMergeChunk;
    __syncthreads();  // the previous item's chunk is no longer read
    if (tid == 0) n_live = 0;
    __syncthreads();
    if (cb + tid < S) {
      const int64_t j = list ? (int64_t)list[cb + tid] : cb + tid;
      if (list || flags[j]) {
        const int at = atomicAdd(&n_live, 1);
        pts[at] = V{a[j], b[j], c[j], T(0)};
      }
    }
    __syncthreads();
    const int live = n_live;
    if (s < S && live > 0) {
      const int64_t i = list ? (int64_t)list[s] : s;
      if (list || flags[i]) {
        const T ia = a[i], ib = b[i], ic = c[i];
        bool dom = false;
        int k = 0;
        for (; k + 4 <= live && !dom; k += 4) {
          const V p0 = pts[k], p1 = pts[k + 1], p2 = pts[k + 2], p3 = pts[k + 3];
          dom = dominates(p0.x, p0.y, p0.z, ia, ib, ic) || dominates(p1.x, p1.y, p1.z, ia, ib, ic) ||
                dominates(p2.x, p2.y, p2.z, ia, ib, ic) || dominates(p3.x, p3.y, p3.z, ia, ib, ic);
        }
        for (; k < live && !dom; ++k) dom = dominates(pts[k].x, pts[k].y, pts[k].z, ia, ib, ic);
        if (dom) flags[i] = 0;
      }
    }
  }
}

__global__ __launch_bounds__(kMaceThreads) void zero_i32_kernel(int32_t* p) {
  if (threadIdx.x == 0) p[0] = 0;
}

__global__ __launch_bounds__(kMaceThreads) void count_flags_kernel(const uint8_t* __restrict__ f, int64_t n,
                                                                   int32_t* __restrict__ out) {
  int cnt = 0;
  for (int64_t i = (int64_t)blockIdx.x * kMaceThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kMaceThreads)
    cnt += f[i] != 0;
  for (int m = 32; m >= 1; m >>= 1) cnt += __shfl_xor(cnt, m);
  if ((threadIdx.x & 63) == 0 && cnt) atomicAdd(out, cnt);
}

namespace {
int device_cus() {
  int dev = 0, cus = 256;
  (void)hipGetDevice(&dev);
  (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  return cus;
}

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

template <typename T>
int run_pareto(const T* a, const T* b, const T* c, const uint8_t* mask, int64_t n, uint8_t* flags,
               int32_t* n_front, hipStream_t s) {
  const int64_t tiles = (n + kParetoTile - 1) / kParetoTile;
  const int64_t P = tiles * kPivotsPerTile;
  // scratch: counts (survivors, pivot front) | list [n] | pa pb pc [P] | pivot flags [P] | packed front [P]
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align256(bytes);
    return at;
  };
  typedef typename Vec4<T>::type V;
  const size_t o_cnt = take(8), o_list = take((size_t)n * 4), o_pa = take((size_t)P * sizeof(T)),
               o_pb = take((size_t)P * sizeof(T)), o_pc = take((size_t)P * sizeof(T)), o_pf = take((size_t)P),
               o_fr = take((size_t)P * sizeof(V));
  unsigned char* ws = (unsigned char*)device_scratch(off, 4);
  if (!ws) return fail(SCOOT_ERR_NO_MEMORY, "pareto: scratch allocation failed");
  int32_t* count = reinterpret_cast<int32_t*>(ws + o_cnt);
  int32_t* list = reinterpret_cast<int32_t*>(ws + o_list);
  T* pa = reinterpret_cast<T*>(ws + o_pa);
  T* pb = reinterpret_cast<T*>(ws + o_pb);
  T* pc = reinterpret_cast<T*>(ws + o_pc);
  uint8_t* pfront = ws + o_pf;
  V* front = reinterpret_cast<V*>(ws + o_fr);
  const int64_t pb_ = (P + kMaceThreads - 1) / kMaceThreads, pc_ = (P + kMergeChunk - 1) / kMergeChunk;
  const int64_t grid_p = std::max<int64_t>(1, std::min<int64_t>(pb_ * pc_, (int64_t)device_cus() * 4));
  const int64_t grid_d = std::min<int64_t>((n + kMaceThreads - 1) / kMaceThreads, (int64_t)device_cus() * 4);
  // A (also zeroes both counts), B, B', C, D
  hipLaunchKernelGGL((pareto_pivot_kernel<T>), dim3((unsigned)tiles), dim3(kMaceThreads), 0, s, a, b, c, mask, n, pa,
                     pb, pc, pfront, count);
  hipLaunchKernelGGL((pareto_merge_kernel<T>), dim3((unsigned)grid_p), dim3(kMaceThreads), 0, s, (const T*)pa,
                     (const T*)pb, (const T*)pc, (const int32_t*)nullptr, (const int32_t*)nullptr, P, pfront);
  hipLaunchKernelGGL((pareto_gather_kernel<T>), dim3((unsigned)pb_), dim3(kMaceThreads), 0, s, (const T*)pa,
                     (const T*)pb, (const T*)pc, (const uint8_t*)pfront, P, front, count);
  hipLaunchKernelGGL((pareto_filter_kernel<T>), dim3((unsigned)tiles), dim3(kMaceThreads), 0, s, a, b, c, mask, n,
                     (const V*)front, flags, list, count);
  hipLaunchKernelGGL((pareto_merge_kernel<T>), dim3((unsigned)grid_d), dim3(kMaceThreads), 0, s, a, b, c,
                     (const int32_t*)list, (const int32_t*)count, (int64_t)0, flags);
  if (n_front) {
    hipLaunchKernelGGL(zero_i32_kernel, dim3(1), dim3(kMaceThreads), 0, s, n_front);
    const int64_t grid3 = std::min<int64_t>((n + kMaceThreads - 1) / kMaceThreads, 1024);
    hipLaunchKernelGGL(count_flags_kernel, dim3((unsigned)grid3), dim3(kMaceThreads), 0, s, (const uint8_t*)flags,
                       n, n_front);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("pareto launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}
}  // namespace

int launch_mace_scores(const void* mu, const void* sigma, int64_t n, scoot_dtype dt, double c, double beta, void* ucb,
                       void* pi, void* ei, void* stream) {
  if (n == 0) return SCOOT_OK;
  hipStream_t s = (hipStream_t)stream;
  const int64_t blocks = std::min<int64_t>((n + kMaceThreads - 1) / kMaceThreads, 4096);
  if (dt == SCOOT_F32)
    hipLaunchKernelGGL(mace_scores_kernel<float>, dim3((unsigned)blocks), dim3(kMaceThreads), 0, s,
                       (const float*)mu, (const float*)sigma, n, (float)c, (float)beta, (float*)ucb, (float*)pi,
                       (float*)ei);
  else
    hipLaunchKernelGGL(mace_scores_kernel<double>, dim3((unsigned)blocks), dim3(kMaceThreads), 0, s,
                       (const double*)mu, (const double*)sigma, n, c, beta, (double*)ucb, (double*)pi, (double*)ei);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("mace launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}

int launch_pareto_front3(const void* a, const void* b, const void* c, const uint8_t* mask, int64_t n, scoot_dtype dt,
                         uint8_t* front, int32_t* n_front, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  if (n == 0) {
    if (n_front) hipLaunchKernelGGL(zero_i32_kernel, dim3(1), dim3(kMaceThreads), 0, s, n_front);
    hipError_t err = hipGetLastError();
    return err == hipSuccess ? SCOOT_OK : fail(SCOOT_ERR_DEVICE, std::string("pareto: ") + hipGetErrorString(err));
  }
  if (dt == SCOOT_F32)
    return run_pareto<float>((const float*)a, (const float*)b, (const float*)c, mask, n, front, n_front, s);
  return run_pareto<double>((const double*)a, (const double*)b, (const double*)c, mask, n, front, n_front, s);
}

}  // namespace scoot
