// Masked top-q selection (Sec. 4.6): the q eligible candidates with the
// largest score, score descending, lowest index first on ties.
//
// Every candidate becomes one integer key whose unsigned order is exactly that
// order: the score's bits mapped to an order-preserving unsigned integer
// (after -0 -> +0), followed by the bit-inverted index.  Key 0 marks an
// ineligible candidate (mask 0 or NaN score); no eligible key is 0.  fp32
// scores fit score and index in one 64-bit key; fp64 scores use a pair.
//
// Stage 1: every wave walks its share of the array in chunks of 1024 keys (16
// per lane) and keeps a running best-q list in its lanes: q rounds of a
// wave-wide argmax (butterfly of shuffles, no barriers) over the chunk plus
// the list.  Stage 2: one workgroup with a wave per chunk of the stage-1
// lists (at most kSel2Waves) runs the same selection over them; with more
// than one wave, the first selects again over the waves' lists (at most one
// chunk).  It writes indices, scores and the count.  Selection is exact integer work, so the result does not
// depend on the grid shape or on the order in which waves run.
//
// The same two stages make the random pick of the MACE suggestion (Sec. 4.5.1,
// Sec. 4.6): candidate i's key is (u_i, inverted index), u_i the i-th output of
// SplitMix64 started from the caller's seed, so the pick is the q flagged
// candidates with the largest draws -- a uniformly random q-subset of the
// flagged set in random order.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>

#include "internal.h"
#include "select.h"

namespace scoot {

// Key sources for stage 1: load(i) reads what key i needs (no branches),
// key(raw, i) forms it.
template <typename T, bool MASKED>
struct ScoreKeys {
  const T* __restrict__ score;
  const uint8_t* __restrict__ mask;  // read only when MASKED
  struct Raw {
    T s;
    uint8_t m;
  };
  __device__ Raw load(int64_t i) const { return Raw{score[i], MASKED ? mask[i] : (uint8_t)1}; }
  __device__ auto key(const Raw& r, int64_t i) const { return make_key(r.s, i, r.m != 0); }
};

// SplitMix64 (Steele, Lea and Flood, OOPSLA 2014; Stafford's finaliser):
// output number i of the generator started from `seed`.
__device__ inline uint64_t splitmix64(uint64_t seed, uint64_t i) {
  uint64_t z = seed + (i + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
struct DrawKeys {
  const uint8_t* __restrict__ flags;
  uint64_t seed;
  typedef uint8_t Raw;
  __device__ Raw load(int64_t i) const { return flags[i]; }
  __device__ Key128 key(Raw f, int64_t i) const {
    const uint64_t u = splitmix64(seed, (uint64_t)i);
    return f ? Key128{u, ~(uint64_t)i} : Key128{0, 0};
  }
};

// part_keys [waves * q], part_count [waves]: each wave's list and its count
// of eligible keys; wave w takes chunks w, w + W, ... (W waves in the grid).
template <typename K, typename Src>
__global__ __launch_bounds__(kSelThreads) void topq_stage1(const Src src, int64_t n, int q, K* __restrict__ part_keys,
                                                           int32_t* __restrict__ part_count) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * (kSelThreads / 64) + (threadIdx.x >> 6);
  const int64_t waves = (int64_t)gridDim.x * (kSelThreads / 64);
  K list{};
  int32_t valid = 0;
  for (int64_t base = wave * kSelChunk; base < n; base += waves * kSelChunk) {
    // Every load is issued before any is used: the index is clamped and a
    // key past the end is zeroed afterwards (no branch around the loads).
    typename Src::Raw raw[kSelPer];
#pragma unroll
    for (int j = 0; j < kSelPer; ++j) {
      const int64_t i = base + (int64_t)j * 64 + lane;
      raw[j] = src.load(i < n ? i : n - 1);
    }
    K keys[kSelPer];
#pragma unroll
    for (int j = 0; j < kSelPer; ++j) {
      const int64_t i = base + (int64_t)j * 64 + lane;
      keys[j] = src.key(raw[j], i);
      if (i >= n) keys[j] = K{};
      valid += keys[j].zero() ? 0 : 1;
    }
    wave_select<K>(keys, list, q);
  }
  for (int m = 32; m >= 1; m >>= 1) valid += __shfl_xor(valid, m);
  if (lane < q) part_keys[wave * q + lane] = list;
  if (lane == 0) part_count[wave] = valid;
}

// One workgroup of W waves: the best q of all stage-1 lists (wave w takes
// chunks w, w + W, ... of them; wave 0 then merges the waves' lists), then
// indices, scores and the count.
template <typename T, typename K>
__global__ __launch_bounds__(64 * kSel2Waves) void topq_stage2(const T* __restrict__ score, int n_parts, int q,
                                                               const K* __restrict__ part_keys,
                                                               const int32_t* __restrict__ part_count,
                                                               int64_t* __restrict__ idx, T* __restrict__ score_out,
                                                               int32_t* __restrict__ n_valid) {
  __shared__ K wave_lists[kSel2Waves * 64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  // the eligible count first: its loads are in flight during the selection
  int32_t count = 0;
  if (n_valid && wave == 0)
    for (int b = lane; b < n_parts; b += 64) count += part_count[b];
  K list{};
  const int64_t total = (int64_t)n_parts * q;
  const int W = blockDim.x >> 6;
  for (int64_t base = (int64_t)wave * kSelChunk; base < total; base += (int64_t)W * kSelChunk) {
    K keys[kSelPer];
#pragma unroll
    for (int j = 0; j < kSelPer; ++j) {
      const int64_t i = base + (int64_t)j * 64 + lane;
      keys[j] = part_keys[i < total ? i : total - 1];
    }
#pragma unroll
    for (int j = 0; j < kSelPer; ++j)
      if (base + (int64_t)j * 64 + lane >= total) keys[j] = K{};
    wave_select<K>(keys, list, q);
  }
  if (W > 1) {
    if (lane < q) wave_lists[wave * q + lane] = list;
    __syncthreads();
    if (wave != 0) return;
    K keys[kSelPer];
#pragma unroll
    for (int j = 0; j < kSelPer; ++j) {
      const int i = j * 64 + lane;
      keys[j] = i < W * q ? wave_lists[i] : K{};
    }
    list = K{};
    wave_select<K>(keys, list, q);
  }
  if (lane < q) {
    if (list.zero()) {
      idx[lane] = -1;
      if (score_out) score_out[lane] = (T)NAN;
    } else {
      const int64_t i = key_index(list);
      idx[lane] = i;
      // the key carries the score; only a zero (which may have been -0) is read back
      if (score_out) {
        const T v = key_score(list);
        score_out[lane] = v == T(0) ? score[i] : v;
      }
    }
  }
  if (n_valid) {  // sum of the stage-1 counts
    for (int m = 32; m >= 1; m >>= 1) count += __shfl_xor(count, m);
    if (lane == 0) *n_valid = count;
  }
}

namespace {
// Stage-1 waves for n keys and q picks: as many as chunks, bounded so that
// stage 2 reads at most kSelMaxKeys2 keys; whole workgroups of four waves.
int64_t select_waves(int64_t n, int q) {
  int64_t waves = (n + kSelChunk - 1) / kSelChunk;
  waves = std::max<int64_t>(1, std::min<int64_t>(waves, std::max(4, kSelMaxKeys2 / q)));
  return (waves + 3) / 4 * 4;
}
// Bytes of the stage-1 lists and counts.
template <typename K>
size_t select_scratch_bytes(int64_t n, int q) {
  const int64_t waves = select_waves(n, q);
  return (size_t)waves * q * sizeof(K) + (size_t)waves * 4;
}

// Launches both stages with the stage-1 lists in ws (at least
// select_scratch_bytes<K>(n, q) bytes of device memory).  score / score_out
// may be null (the random pick writes indices only).
template <typename T, typename K, typename Src>
hipError_t run_select(const Src& src, const T* score, int64_t n, int q, int64_t* idx, T* score_out,
                      int32_t* n_valid, unsigned char* ws, hipStream_t s) {
  const int64_t waves = select_waves(n, q);
  const size_t kbytes = (size_t)waves * q * sizeof(K);
  K* pk = reinterpret_cast<K*>(ws);
  int32_t* pc = reinterpret_cast<int32_t*>(ws + kbytes);
  hipLaunchKernelGGL((topq_stage1<K, Src>), dim3((unsigned)(waves / 4)), dim3(kSelThreads), 0, s, src, n, q, pk, pc);
  const int w2 = (int)std::min<int64_t>(kSel2Waves, (waves * q + kSelChunk - 1) / kSelChunk);
  hipLaunchKernelGGL((topq_stage2<T, K>), dim3(1), dim3(64 * w2), 0, s, score, (int)waves, q, pk, pc, idx,
                     score_out, n_valid);
  return hipGetLastError();
}

// As run_select, with the stage-1 lists in the library's grow-only scratch.
template <typename T, typename K, typename Src>
int run_select_scratch(const Src& src, const T* score, int64_t n, int q, int64_t* idx, T* score_out,
                       int32_t* n_valid, hipStream_t s) {
  unsigned char* ws = (unsigned char*)device_scratch(select_scratch_bytes<K>(n, q), 3);
  if (!ws) return fail(SCOOT_ERR_NO_MEMORY, "topq: scratch allocation failed");
  const hipError_t err = run_select<T, K>(src, score, n, q, idx, score_out, n_valid, ws, s);
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("topq launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}
}  // namespace

int launch_topq(const void* score, const uint8_t* mask, int64_t n, scoot_dtype dt, int q, int64_t* idx,
                void* score_out, int32_t* n_valid, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  if (dt == SCOOT_F32) {
    if (mask)
      return run_select_scratch<float, Key64>(ScoreKeys<float, true>{(const float*)score, mask}, (const float*)score,
                                              n, q, idx, (float*)score_out, n_valid, s);
    return run_select_scratch<float, Key64>(ScoreKeys<float, false>{(const float*)score, mask}, (const float*)score,
                                            n, q, idx, (float*)score_out, n_valid, s);
  }
  if (mask)
    return run_select_scratch<double, Key128>(ScoreKeys<double, true>{(const double*)score, mask},
                                              (const double*)score, n, q, idx, (double*)score_out, n_valid, s);
  return run_select_scratch<double, Key128>(ScoreKeys<double, false>{(const double*)score, mask},
                                            (const double*)score, n, q, idx, (double*)score_out, n_valid, s);
}

int launch_topq_stage2(const void* score, scoot_dtype dt, int n_parts, int q, const void* part_keys,
                       const int32_t* part_count, int64_t* idx, void* score_out, int32_t* n_valid, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const int w2 = (int)std::min<int64_t>(kSel2Waves, ((int64_t)n_parts * q + kSelChunk - 1) / kSelChunk);
  if (dt == SCOOT_F32)
    hipLaunchKernelGGL((topq_stage2<float, Key64>), dim3(1), dim3(64 * w2), 0, s, (const float*)score, n_parts, q,
                       (const Key64*)part_keys, part_count, idx, (float*)score_out, n_valid);
  else
    hipLaunchKernelGGL((topq_stage2<double, Key128>), dim3(1), dim3(64 * w2), 0, s, (const double*)score, n_parts,
                       q, (const Key128*)part_keys, part_count, idx, (double*)score_out, n_valid);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("topq launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}

int launch_random_pick(const uint8_t* flags, int64_t n, uint64_t seed, int q, int64_t* idx, int32_t* n_flagged,
                       void* stream) {
  const DrawKeys src{flags, seed};
  return run_select_scratch<double, Key128>(src, (const double*)nullptr, n, q, idx, (double*)nullptr, n_flagged,
                                            (hipStream_t)stream);
}

// ---------------------------------------------------------------------------
// Top-q without any allocation, for callers that cannot allocate device
// memory.  The stage-1 lists live in `scratch`, one fixed array per GPU that
// stays allocated until the process ends.  The largest need over every
// n < 2^31 and 1 <= q <= SCOOT_MAX_Q is 327,680 bytes (q = 1, fp64 keys: 16384
// waves x (16 + 4) bytes); the array is that size.  Stage 1 writes every list
// entry and count stage 2 reads, so nothing needs clearing between calls;
// calls that overlap on one GPU share the array and race.
constexpr size_t kTopqStaticBytes = 327680;
static __device__ __align__(256) unsigned char scratch[kTopqStaticBytes];

namespace {
constexpr int kStaticMaxDevices = 64;
std::mutex g_static_mu;
unsigned char* g_static_ptr[kStaticMaxDevices] = {};

// The device address of `scratch` on the current device, looked up on the
// first call on that device (with it current) and kept: the host-side name
// of a __device__ array is not a device address.
int static_scratch(unsigned char** out) {
  int d = -1;
  if (hipGetDevice(&d) != hipSuccess || d < 0 || d >= kStaticMaxDevices)
    return fail_static(SCOOT_ERR_DEVICE, "topq (no allocation): no usable current device");
  std::lock_guard<std::mutex> lk(g_static_mu);
  if (!g_static_ptr[d]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p)
      return fail_static(SCOOT_ERR_DEVICE, "topq (no allocation): cannot resolve the scratch array's address");
    g_static_ptr[d] = (unsigned char*)p;
  }
  *out = g_static_ptr[d];
  return SCOOT_OK;
}
}  // namespace

int launch_topq_static(const void* score, const uint8_t* mask, int64_t n, scoot_dtype dt, int q, int64_t* idx,
                       void* score_out, int32_t* n_valid, void* stream) {
  const size_t need = dt == SCOOT_F32 ? select_scratch_bytes<Key64>(n, q) : select_scratch_bytes<Key128>(n, q);
  if (need > kTopqStaticBytes)
    return fail_static(SCOOT_ERR_UNSUPPORTED, "topq (no allocation): the stage-1 lists exceed the scratch array");
  unsigned char* ws = nullptr;
  const int rc = static_scratch(&ws);
  if (rc != SCOOT_OK) return rc;
  hipStream_t s = (hipStream_t)stream;
  hipError_t err;
  if (dt == SCOOT_F32) {
    err = mask ? run_select<float, Key64>(ScoreKeys<float, true>{(const float*)score, mask}, (const float*)score, n, q,
                                          idx, (float*)score_out, n_valid, ws, s)
               : run_select<float, Key64>(ScoreKeys<float, false>{(const float*)score, mask}, (const float*)score, n,
                                          q, idx, (float*)score_out, n_valid, ws, s);
  } else {
    err = mask ? run_select<double, Key128>(ScoreKeys<double, true>{(const double*)score, mask},
                                            (const double*)score, n, q, idx, (double*)score_out, n_valid, ws, s)
               : run_select<double, Key128>(ScoreKeys<double, false>{(const double*)score, mask},
                                            (const double*)score, n, q, idx, (double*)score_out, n_valid, ws, s);
  }
  if (err != hipSuccess) return fail_static(SCOOT_ERR_DEVICE, "topq (no allocation): kernel launch failed");
  return SCOOT_OK;
}

}  // namespace scoot
