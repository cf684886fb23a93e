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
// Front, two stages:
//  1. tiles of 1024 candidates, one per workgroup: the tile's eligible
//     members are compacted into LDS and each candidate is checked against
//     all of them; survivors set their flag and append their index to a list
//     (one global atomic per wave for the space);
//  2. every survivor is checked against all survivors, staged through LDS in
//     chunks; dominated survivors clear their flag.
// This is exact: domination is transitive on a finite set, so whatever is
// dominated is dominated by a front member, and front members survive stage 1.
// The flags do not depend on the order of the list.  Cost: n x 1024
// comparisons in stage 1 (each wave stops at its lanes' first dominator) and
// S^2 in stage 2, S = survivors of stage 1 (a few per tile when the three
// scores agree; up to n when they are in full conflict).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "internal.h"
#include "normal.h"

namespace scoot {

constexpr int kMaceThreads = 256;
constexpr int kParetoTile = 1024;   // candidates per stage-1 workgroup, 4 per thread
constexpr int kParetoChunk = 1024;  // survivors staged in LDS per stage-2 step

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

template <typename T>
__global__ __launch_bounds__(kMaceThreads) void pareto_tile_kernel(const T* __restrict__ a, const T* __restrict__ b,
                                                                   const T* __restrict__ c,
                                                                   const uint8_t* __restrict__ mask, int64_t n,
                                                                   uint8_t* __restrict__ flags,
                                                                   int32_t* __restrict__ list,
                                                                   int32_t* __restrict__ count) {
  __shared__ T sa[kParetoTile], sb[kParetoTile], sc[kParetoTile];
  __shared__ int n_live;
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t base = (int64_t)blockIdx.x * kParetoTile;
  if (tid == 0) n_live = 0;
  __syncthreads();
  T va[4], vb[4], vc[4];
  bool ok[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t i = base + r * kMaceThreads + tid;
    ok[r] = false;
    va[r] = vb[r] = vc[r] = T(0);
    if (i < n) {
      va[r] = a[i];
      vb[r] = b[i];
      vc[r] = c[i];
      ok[r] = (!mask || mask[i] != 0) && va[r] == va[r] && vb[r] == vb[r] && vc[r] == vc[r];
    }
    if (ok[r]) {  // the tile's eligible members, in any order
      const int at = atomicAdd(&n_live, 1);
      sa[at] = va[r];
      sb[at] = vb[r];
      sc[at] = vc[r];
    }
  }
  __syncthreads();
  const int live = n_live;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t i = base + r * kMaceThreads + tid;
    bool surv = ok[r];
    if (surv)
      for (int j = 0; j < live; ++j)
        if (dominates(sa[j], sb[j], sc[j], va[r], vb[r], vc[r])) {
          surv = false;
          break;
        }
    if (i < n) flags[i] = surv ? 1 : 0;
    const uint64_t bal = __ballot(surv);
    if (bal) {
      int at = 0;
      if (lane == 0) at = atomicAdd(count, (int)__popcll(bal));
      at = __shfl(at, 0);
      const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
      if (surv) list[at + below] = (int32_t)i;
    }
  }
}

template <typename T>
__global__ __launch_bounds__(kMaceThreads) void pareto_merge_kernel(const T* __restrict__ a, const T* __restrict__ b,
                                                                    const T* __restrict__ c,
                                                                    const int32_t* __restrict__ list,
                                                                    const int32_t* __restrict__ count,
                                                                    uint8_t* __restrict__ flags) {
  __shared__ T sa[kParetoChunk], sb[kParetoChunk], sc[kParetoChunk];
  const int tid = threadIdx.x;
  const int S = *count;
  for (int64_t s0 = (int64_t)blockIdx.x * kMaceThreads; s0 < S; s0 += (int64_t)gridDim.x * kMaceThreads) {
    const int64_t sidx = s0 + tid;
    const bool mine = sidx < S;
    int32_t i = 0;
    T ia = T(0), ib = T(0), ic = T(0);
    if (mine) {
      i = list[sidx];
      ia = a[i];
      ib = b[i];
      ic = c[i];
    }
    bool alive = mine;
    for (int cb = 0; cb < S; cb += kParetoChunk) {
      __syncthreads();  // the previous chunk is no longer read
      const int cnt = S - cb < kParetoChunk ? S - cb : kParetoChunk;
      for (int k = tid; k < cnt; k += kMaceThreads) {
        const int32_t j = list[cb + k];
        sa[k] = a[j];
        sb[k] = b[j];
        sc[k] = c[j];
      }
      __syncthreads();
      if (alive)
        for (int k = 0; k < cnt; ++k)
          if (dominates(sa[k], sb[k], sc[k], ia, ib, ic)) {
            alive = false;
            break;
          }
      if (!__syncthreads_or(alive)) break;  // every survivor of this batch is dominated
    }
    if (mine && !alive) flags[i] = 0;
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

template <typename T>
int run_pareto(const T* a, const T* b, const T* c, const uint8_t* mask, int64_t n, uint8_t* flags,
               int32_t* n_front, hipStream_t s) {
  // scratch: survivor count, then the survivor list (capacity n)
  unsigned char* ws = (unsigned char*)device_scratch(256 + (size_t)n * 4, 4);
  if (!ws) return fail(SCOOT_ERR_NO_MEMORY, "pareto: scratch allocation failed");
  int32_t* count = reinterpret_cast<int32_t*>(ws);
  int32_t* list = reinterpret_cast<int32_t*>(ws + 256);
  hipLaunchKernelGGL(zero_i32_kernel, dim3(1), dim3(kMaceThreads), 0, s, count);
  const int64_t tiles = (n + kParetoTile - 1) / kParetoTile;
  hipLaunchKernelGGL((pareto_tile_kernel<T>), dim3((unsigned)tiles), dim3(kMaceThreads), 0, s, a, b, c, mask, n,
                     flags, list, count);
  const int64_t grid2 = std::min<int64_t>((n + kMaceThreads - 1) / kMaceThreads, (int64_t)device_cus() * 8);
  hipLaunchKernelGGL((pareto_merge_kernel<T>), dim3((unsigned)grid2), dim3(kMaceThreads), 0, s, a, b, c,
                     (const int32_t*)list, (const int32_t*)count, flags);
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
