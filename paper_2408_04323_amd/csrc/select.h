// Integer keys and wave-level selection shared by the top-q kernels and the
// acquisition kernel that forms keys in its epilogue (Sec. 4.6: the q
// eligible candidates with the largest score, lowest index first on ties).
//
// A key's unsigned order is exactly that order: the score's bits mapped to an
// order-preserving unsigned integer (after -0 -> +0), then the bit-inverted
// index.  Key 0 marks an ineligible candidate (mask 0 or NaN score).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace scoot {

constexpr int kSelThreads = 256;  // stage 1 workgroup: four independent waves
constexpr int kSelPer = 16;       // keys per lane per chunk
constexpr int kSelChunk = 64 * kSelPer;
constexpr int kSelMaxKeys2 = 16384;  // bound on the stage-1 lists stage 2 reads (waves x q)
constexpr int kSel2Waves = 16;       // stage 2 workgroup; kSel2Waves x q (q <= 64) keys fit one chunk

struct Key64 {
  uint64_t v;
  __device__ bool operator>(const Key64& o) const { return v > o.v; }
  __device__ bool zero() const { return v == 0; }
};
struct Key128 {
  uint64_t hi, lo;
  __device__ bool operator>(const Key128& o) const { return hi > o.hi || (hi == o.hi && lo > o.lo); }
  __device__ bool zero() const { return hi == 0 && lo == 0; }
};

// Branch-free, so that a thread's loads can all be in flight before any key
// is formed.
__device__ inline Key64 make_key(float s, int64_t i, bool ok) {
  uint32_t b = __float_as_uint(s + 0.0f);
  b = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  const uint64_t k = ((uint64_t)b << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)i);
  return Key64{ok && s == s ? k : 0ull};
}
__device__ inline Key128 make_key(double s, int64_t i, bool ok) {
  uint64_t b = (uint64_t)__double_as_longlong(s + 0.0);
  b = (b & 0x8000000000000000ull) ? ~b : (b | 0x8000000000000000ull);
  const bool keep = ok && s == s;
  return Key128{keep ? b : 0ull, keep ? ~(uint64_t)i : 0ull};
}
__device__ inline int64_t key_index(const Key64& k) { return (int64_t)(0xFFFFFFFFu - (uint32_t)k.v); }
__device__ inline int64_t key_index(const Key128& k) { return (int64_t)(~k.lo); }
// The score a non-zero key was formed from (the inverse of the bit mapping;
// -0 comes back as +0).
__device__ inline float key_score(const Key64& k) {
  const uint32_t b = (uint32_t)(k.v >> 32);
  return __uint_as_float((b & 0x80000000u) ? (b & 0x7FFFFFFFu) : ~b);
}
__device__ inline double key_score(const Key128& k) {
  const uint64_t b = k.hi;
  return __longlong_as_double((long long)((b & 0x8000000000000000ull) ? (b & 0x7FFFFFFFFFFFFFFFull) : ~b));
}

// Wave-wide maximum of a key, returned in every lane (uniform).  Inside each
// row of 16 lanes four DPP exchanges (quad permutations, then the half-row
// and row mirrors) leave the row's maximum in all of its lanes; the four row
// maxima are then read out and combined.  DPP moves and lane reads are plain
// vector/scalar instructions: no trip through the LDS crossbar per step.
template <int CTRL>
__device__ inline uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
__device__ inline uint32_t readlane_u32(uint32_t v, int l) { return (uint32_t)__builtin_amdgcn_readlane((int)v, l); }

template <int CTRL>
__device__ inline Key64 dpp_key(const Key64& k) {
  const uint32_t lo = (uint32_t)k.v, hi = (uint32_t)(k.v >> 32);
  return Key64{((uint64_t)dpp_u32<CTRL>(hi) << 32) | dpp_u32<CTRL>(lo)};
}
template <int CTRL>
__device__ inline Key128 dpp_key(const Key128& k) {
  const uint64_t hi = ((uint64_t)dpp_u32<CTRL>((uint32_t)(k.hi >> 32)) << 32) | dpp_u32<CTRL>((uint32_t)k.hi);
  const uint64_t lo = ((uint64_t)dpp_u32<CTRL>((uint32_t)(k.lo >> 32)) << 32) | dpp_u32<CTRL>((uint32_t)k.lo);
  return Key128{hi, lo};
}
__device__ inline Key64 readlane_key(const Key64& k, int l) {
  return Key64{((uint64_t)readlane_u32((uint32_t)(k.v >> 32), l) << 32) | readlane_u32((uint32_t)k.v, l)};
}
__device__ inline Key128 readlane_key(const Key128& k, int l) {
  return Key128{((uint64_t)readlane_u32((uint32_t)(k.hi >> 32), l) << 32) | readlane_u32((uint32_t)k.hi, l),
                ((uint64_t)readlane_u32((uint32_t)(k.lo >> 32), l) << 32) | readlane_u32((uint32_t)k.lo, l)};
}
template <typename K>
__device__ inline K key_max(const K& a, const K& b) {
  return a > b ? a : b;
}
constexpr int kDppQuadXor1 = 0xB1;   // quad_perm [1, 0, 3, 2]
constexpr int kDppQuadXor2 = 0x4E;   // quad_perm [2, 3, 0, 1]
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;

template <typename K>
__device__ inline K wave_max_key(K k) {
  k = key_max(k, dpp_key<kDppQuadXor1>(k));
  k = key_max(k, dpp_key<kDppQuadXor2>(k));
  k = key_max(k, dpp_key<kDppRowHalfMirror>(k));
  k = key_max(k, dpp_key<kDppRowMirror>(k));
  return key_max(key_max(readlane_key(k, 0), readlane_key(k, 16)), key_max(readlane_key(k, 32), readlane_key(k, 48)));
}

// q rounds of wave argmax over the lane's PER keys plus the running list
// (lane r < q holds entry r, zero = empty).  Rewrites the list.  Rounds stop
// once no key is left.
template <typename K, int PER = kSelPer>
__device__ void wave_select(K (&keys)[PER], K& list, int q) {
  const int lane = threadIdx.x & 63;
  K extra = list, next{};
  for (int r = 0; r < q; ++r) {
    K best = extra;
#pragma unroll
    for (int j = 0; j < PER; ++j)
      if (keys[j] > best) best = keys[j];
    best = wave_max_key(best);  // the same in every lane
    if (best.zero()) break;
    // remove it from its owner (keys are unique)
    if (!(extra > best) && !(best > extra)) extra = K{};
#pragma unroll
    for (int j = 0; j < PER; ++j)
      if (!(keys[j] > best) && !(best > keys[j])) keys[j] = K{};
    if (lane == r) next = best;
  }
  list = next;
}

// The list's entry r (zero when the list holds fewer), in every lane; r must
// be the same in every lane.
__device__ inline Key64 list_entry(const Key64& list, int r) { return readlane_key(list, r); }
__device__ inline Key128 list_entry(const Key128& list, int r) { return readlane_key(list, r); }

}  // namespace scoot
