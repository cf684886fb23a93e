// GP posterior over a candidate pool (Sec. 4.3, Eq. 4-5), fused:
//
//   K*[c, i] = k(x_c, X_i)                     Matern-5/2 ARD, generated on chip
//   mu[c]    = c0 + sum_i K*[c, i] alpha_i      (Eq. 4)
//   V        = L^-1 K*^T                         triangular product on matrix cores
//   sigma[c] = sqrt(max(0, s2 - sum_i V[i, c]^2))   (Eq. 5, latent f)
//   ei[c]    = G(best + xi)   optional fused EI epilogue (Eq. 8)
//
// One workgroup owns a tile of candidates (64 in fp32, 32 in fp64) and runs
// three phases:
//   1. generate: every wave computes K* for a share of the observation rows,
//      for all candidates of the tile, straight into LDS in the B-operand
//      order of the MFMA instruction; alpha is folded in on the way (mu);
//   2. multiply: every wave takes whole row blocks I of V (a per-SIMD row plan
//      keeps the triangular work balanced), accumulates sum_{J<=I} Linv[I,J] K*[J]
//      on the matrix cores (A from the packed L^-1 in L2, B from LDS), and
//      keeps only the squared norms of its rows;
//   3. reduce: partial norms and means of all waves are summed per candidate.
// K* and V never touch HBM.  L^-1 is shared by every workgroup (L2-resident).
//
// Covariance with folded constants: with per-dimension scale
// w_k = sqrt5 * log2(e) / l_k, u = sqrt(sum_k (w_k (x_k - X_ik))^2) equals
// sqrt5 r log2(e), and k = (c0 + u (c1 + u c2)) 2^-u with c0 = s2,
// c1 = s2 ln2, c2 = s2 ln2^2 / 3.  Observations arrive pre-scaled; padding rows
// sit at coordinate 1e4 (fp64) or carry a squared norm of 1e30 (the fp32
// augmented rows), so their covariance underflows to exactly 0, and their
// alpha and L^-1 entries are 0.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <type_traits>
#include <utility>

#include "internal.h"

namespace scoot {

typedef float f4_t __attribute__((ext_vector_type(4)));
typedef float f16_t __attribute__((ext_vector_type(16)));
typedef double d2_t __attribute__((ext_vector_type(2)));
typedef double d4_t __attribute__((ext_vector_type(4)));

// E[(c - Y)^+] for Y ~ N(mu, sd^2), in double (epilogue only).
__device__ inline double partial_expectation_d(double c, double mu, double sd) {
  if (!(sd > 0)) return fmax(c - mu, 0.0);
  double u = (c - mu) / sd;
  return sd * (u * 0.5 * erfc(-u * 0.70710678118654752440) +
               0.39894228040143267794 * exp(-0.5 * u * u));
}

// ---------------------------------------------------------------------------
// fp32.  Everything runs on 16 x 16 MFMA tiles; a candidate tile is 64
// candidates, four column tiles ct of 16.  Lane l has g = l / 16 and
// c = l % 16.
//
// Phase 1, squared distances on the fp64 matrix cores: with augmented rows
// A_i = (2 X_i, -|X_i|^2, -1) for the observations and B_x = (x, 1, |x|^2)
// for the candidates (scaled coordinates, fp64), A_i . B_x = -|x - X_i|^2, so
// one v_mfma_f64_16x16x4f64 chain over ceil((d + 2) / 4) steps gives -u^2
// for 16 observations x 16 candidates, exact to double rounding (no
// cancellation that float could see).  The observations are packed so that
// output lane l, register r holds observation 16J + 4g + r of candidate c
// (the instruction's own order is row g + 4r there): the lane turns its four values
// into K* in float (sqrt, exp2, the polynomial), folds alpha into the mean,
// and stores them as one float4 -- which is exactly the B operand the
// triangular product reads.
//
// Phase 2, V = L^-1 K*^T on v_mfma_f32_16x16x4f32 over 16 x 16 blocks of the
// triangle (executed work (nb16 + 1) / nb16 of the triangle's, against
// (nb32 + 1) / nb32 for 32 x 32 blocks).  The contraction index of a block is
// ordered k = 4g + s (s the MFMA step), so at step s lane l holds
// L^-1[16I + c][16J + 4g + s] and K*[16J + 4g + s][candidate c] -- the
// float4 phase 1 stored.  Output lane l, register r holds row 16I + 4g + r of
// candidate c.
// ---------------------------------------------------------------------------
struct Post32 {
  int64_t n;
  int d, nb16;
  double scale[SCOOT_MAX_DIM];
  float c0, c1, c2;
  double s2, prior, ei_c;
  RowPlan16 plan;  // 16-row blocks of each wave and where they start in the packed inverse
  int64_t v_ld;    // row stride of a kept V
};

// The 16 MFMA steps of a block: four k-steps for each of the four column
// tiles, the tiles' chains interleaved.  The next block's A (from L2 at
// an_src) is requested first, a block ahead of its use; its B (from LDS at
// bn_src) between the steps, not in one burst before them.
__device__ inline void mfma_block16f(f4_t (&acc)[4], const f4_t& a, const f4_t (&b)[4], f4_t (&bn)[4],
                                     const f4_t* bn_src, f4_t& an, const f4_t* an_src) {
  an = *an_src;
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[ct][0], acc[ct], 0, 0, 0);
  __builtin_amdgcn_sched_barrier(0);
  bn[0] = bn_src[0];
  bn[1] = bn_src[64];
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[ct][1], acc[ct], 0, 0, 0);
  __builtin_amdgcn_sched_barrier(0);
  bn[2] = bn_src[128];
  bn[3] = bn_src[192];
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[ct][2], acc[ct], 0, 0, 0);
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[ct][3], acc[ct], 0, 0, 0);
}
__device__ inline void load_b16f(f4_t (&b)[4], const f4_t* ks, int J, int lane) {
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) b[ct] = ks[(J * 4 + ct) * 64 + lane];
}

// Where V goes when it is kept (the sequential believer needs it): row-major,
// rows = observations in their order, row stride ld.
struct VStore {
  float* v;
  int64_t ld;
  int64_t c0;  // first candidate of the tile
  int64_t n;
};

// Completes a row block: squared norms of its V columns into sq[ct], the
// block itself into V when kept, and clears the accumulators for the next row.
template <bool KEEP_V>
__device__ inline void finish_row16(f4_t (&acc)[4], float (&sq)[4], const VStore& vs, int I, int lane) {
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) {
    float p = 0.0f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float v = acc[ct][r];
      if constexpr (KEEP_V) {
        const int64_t cand = vs.c0 + ct * 16 + (lane & 15);
        const int64_t row = 16 * I + 4 * (lane >> 4) + r;
        if (cand < vs.n) vs.v[row * vs.ld + cand] = v;
      }
      p = fmaf(v, v, p);
    }
    sq[ct] += p;
    acc[ct] = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
  }
}

// One tile's pass over the wave's blocks, one block of read-ahead of both
// operands in two fixed register sets.  The A stream is the same for every
// tile, so its read-ahead wraps: on entry ax holds the wave's first block,
// and on exit it holds it again for the next tile.
template <bool KEEP_V>
__device__ inline void wave_tile16f(const f4_t* __restrict__ ap, const f4_t* ks, uint64_t lo, uint64_t hi, int count,
                                    int lane, f4_t& ax, float (&sq)[4], const VStore& vs) {
  // the accumulators start each row at zero (finish_row16 clears them)
  f4_t acc[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) acc[ct] = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
  constexpr uint64_t kMask = (1u << kRowBits16) - 1;
  int I = (int)(lo & kMask), J = 0;
  auto next_j = [&](int j, int i) { return j == i ? 0 : j + 1; };
  auto advance = [&]() {
    if (J == I) {
      finish_row16<KEEP_V>(acc, sq, vs, I, lane);
      J = 0;
      lo = (lo >> kRowBits16) | (hi << (64 - kRowBits16));
      hi >>= kRowBits16;
      I = (int)(lo & kMask);
    } else {
      ++J;
    }
  };
  f4_t ay, bx[4], by[4];
  load_b16f(bx, ks, 0, lane);
  const f4_t* kl = ks + lane;
  int k = 0;
  for (; k + 1 < count; k += 2) {
    mfma_block16f(acc, ax, bx, by, kl + next_j(J, I) * 256, ay, ap + (size_t)(k + 1) * 64);
    __builtin_amdgcn_sched_barrier(0);
    advance();
    mfma_block16f(acc, ay, by, bx, kl + next_j(J, I) * 256, ax, ap + (size_t)(k + 2 < count ? k + 2 : 0) * 64);
    __builtin_amdgcn_sched_barrier(0);
    advance();
  }
  if (k < count) {
    mfma_block16f(acc, ax, bx, by, kl + next_j(J, I) * 256, ay, ap);
    __builtin_amdgcn_sched_barrier(0);
    advance();
    ax = ay;
  }
}

// Persistent: workgroup g takes tiles g, g + G, g + 2G, ... (G = grid size),
// so the inverse-factor stream and the next tile's coordinates are in flight
// across tile boundaries.  Phase 1: wave w takes the 16-observation blocks
// J = w, w + WAVES, ...  Phase 2: the wave's row blocks from the plan.
// Phase 3: partial norms and means summed per candidate.
template <int WAVES, int D, bool KEEP_V>
__global__ __launch_bounds__(WAVES * 64, 8 / WAVES) void posterior_f32_kernel(
    const float* __restrict__ Xc, const f4_t* __restrict__ linv, const double* __restrict__ xq,
    const float* __restrict__ alpha, float* __restrict__ mu_out, float* __restrict__ sd_out,
    float* __restrict__ ei_out, float* __restrict__ v_out, const Post32 a) {
  constexpr int S = (D + 2 + 3) / 4;  // fp64 MFMA steps of the augmented rows
  extern __shared__ __align__(16) unsigned char smem[];
  f4_t* ks = reinterpret_cast<f4_t*>(smem);  // [nb16][4 ct][64 lanes] float4
  const int nb16 = a.nb16;
  float* sig_red = reinterpret_cast<float*>(ks + (size_t)nb16 * 4 * 64);  // [WAVES][4 ct][16]
  float* mu_red = sig_red + WAVES * 64;                                    // [WAVES][4 ct][16]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int g = lane >> 4, c = lane & 15;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t n_tiles = (a.n + 63) >> 6;

  // Plan entry of this wave.  With 8 waves, entries p and p + 4 are meant to
  // share a SIMD: each wave takes simd + 4 * (its arrival order on the SIMD),
  // unless the workgroup did not land as two waves per SIMD; then entry =
  // wave.  Either way every entry is taken exactly once.
  int p = wave;
  if constexpr (WAVES == 8) {
    int* on_simd = reinterpret_cast<int*>(mu_red + WAVES * 64);  // [4]
    if (tid < 4) on_simd[tid] = 0;
    __syncthreads();
    const int simd = (int)((__builtin_amdgcn_s_getreg((31 << 11) | 4) >> 4) & 3);  // HW_ID.SIMD_ID
    int slot = 0;
    if (lane == 0) slot = atomicAdd(&on_simd[simd], 1);
    slot = __shfl(slot, 0);
    __syncthreads();
    if (on_simd[0] == 2 && on_simd[1] == 2 && on_simd[2] == 2 && on_simd[3] == 2) p = simd + 4 * slot;
    p = __builtin_amdgcn_readfirstlane(p);
  }
  const uint64_t rows_lo = a.plan.lo[p], rows_hi = a.plan.hi[p];
  const int count = a.plan.blk_start[p + 1] - a.plan.blk_start[p];
  const f4_t* ap = linv + (size_t)a.plan.blk_start[p] * 64 + lane;
  f4_t ax = {0.0f, 0.0f, 0.0f, 0.0f};
  if (count > 0) ax = ap[0];

  // The lane's components of the candidates' augmented rows: step s of the
  // cross-term chain reads component k = 4s + g.
  double wk[S];
#pragma unroll
  for (int s = 0; s < S; ++s) wk[s] = 4 * s + g < D ? a.scale[4 * s + g] : 0.0;

  int64_t tile = blockIdx.x;
  float xr[D];  // candidate tile * 64 + lane, for its squared norm
  float xb[4][S];  // component 4s + g of candidate 16 ct + c (raw float)
  auto load_tile = [&](int64_t t) {
    const int64_t own = min(t * 64 + lane, a.n - 1);
#pragma unroll
    for (int q = 0; q < D; ++q) xr[q] = Xc[own * D + q];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      const int64_t cand = min(t * 64 + ct * 16 + c, a.n - 1);
#pragma unroll
      for (int s = 0; s < S; ++s) xb[ct][s] = 4 * s + g < D ? Xc[cand * D + min(4 * s + g, D - 1)] : 0.0f;
    }
  };
  load_tile(tile);

  for (; tile < n_tiles; tile += gridDim.x) {
    const int64_t c0 = tile * 64;
    // squared norm of the lane's own candidate, then the B operands
    double nrm = 0.0;
#pragma unroll
    for (int q = 0; q < D; ++q) {
      const double t = (double)xr[q] * a.scale[q];
      nrm = fma(t, t, nrm);
    }
    double bq[4][S];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      const double nc = __shfl(nrm, ct * 16 + c);
#pragma unroll
      for (int s = 0; s < S; ++s) {
        const int k = 4 * s + g;
        bq[ct][s] = k < D ? (double)xb[ct][s] * wk[s] : (k == D ? 1.0 : (k == D + 1 ? nc : 0.0));
      }
    }
    // next tile's coordinates, in flight during this one
    const int64_t next = tile + gridDim.x;
    if (next < n_tiles) load_tile(next);

    // The K* generation runs at a raised wave priority and the product at
    // the normal one: where the CU's two workgroups are in different phases,
    // the one generating is served first and reaches its product sooner, so
    // that the SIMDs less often wait with both in the same phase (measured:
    // 2-3% less time per launch at m = 256).
    __builtin_amdgcn_s_setprio(2);
    // ---- phase 1: K* of observation blocks J = wave, wave + WAVES, ... ---
    // The block's operands are loaded one block ahead; its four column
    // tiles' chains are issued interleaved (independent accumulators), then
    // their values are turned into K*.
    float mu_part[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    double aq[S];
    f4_t al = {0.0f, 0.0f, 0.0f, 0.0f};
    if (wave < nb16) {
#pragma unroll
      for (int s = 0; s < S; ++s) aq[s] = xq[((size_t)wave * S + s) * 64 + lane];
      al = *reinterpret_cast<const f4_t*>(alpha + 16 * wave + 4 * g);
    }
    for (int J = wave; J < nb16; J += WAVES) {
      d4_t cr[4];
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) cr[ct] = d4_t{0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int s = 0; s < S; ++s)
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) cr[ct] = __builtin_amdgcn_mfma_f64_16x16x4f64(aq[s], bq[ct][s], cr[ct], 0, 0, 0);
      const f4_t alj = al;
      const int Jn = J + WAVES < nb16 ? J + WAVES : J;
#pragma unroll
      for (int s = 0; s < S; ++s) aq[s] = xq[((size_t)Jn * S + s) * 64 + lane];
      al = *reinterpret_cast<const f4_t*>(alpha + 16 * Jn + 4 * g);
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) {
        f4_t kv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float u = __builtin_amdgcn_sqrtf(fmaxf((float)(-cr[ct][r]), 0.0f));
          const float kval = fmaf(u, fmaf(u, a.c2, a.c1), a.c0) * __builtin_amdgcn_exp2f(-u);
          kv[r] = kval;
          mu_part[ct] = fmaf(kval, alj[r], mu_part[ct]);
        }
        ks[(J * 4 + ct) * 64 + lane] = kv;
      }
    }
    __syncthreads();

    __builtin_amdgcn_s_setprio(0);
    // ---- phase 2: this wave's row blocks of V = L^-1 K*^T -----------------
    float sq[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (count > 0) {
      const VStore vs{v_out, a.v_ld, c0, a.n};
      wave_tile16f<KEEP_V>(ap, ks, rows_lo, rows_hi, count, lane, ax, sq, vs);
    }

    // ---- phase 3: reduce over the four lane rows, the waves, write ---------
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      sq[ct] += __shfl_xor(sq[ct], 16);
      sq[ct] += __shfl_xor(sq[ct], 32);
      mu_part[ct] += __shfl_xor(mu_part[ct], 16);
      mu_part[ct] += __shfl_xor(mu_part[ct], 32);
    }
    if (g == 0) {
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) {
        sig_red[(wave * 4 + ct) * 16 + c] = sq[ct];
        mu_red[(wave * 4 + ct) * 16 + c] = mu_part[ct];
      }
    }
    __syncthreads();
    if (tid < 64) {
      const int64_t cand = c0 + tid;
      if (cand < a.n) {
        double ss = 0.0, mm = 0.0;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) {
          ss += (double)sig_red[w * 64 + tid];
          mm += (double)mu_red[w * 64 + tid];
        }
        const double sd = sqrt(fmax(a.s2 - ss, 0.0));
        const double mu = a.prior + mm;
        mu_out[cand] = (float)mu;
        sd_out[cand] = (float)sd;
        if (ei_out) ei_out[cand] = (float)partial_expectation_d(a.ei_c, (double)(float)mu, (double)(float)sd);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// fp64: v_mfma_f64_16x16x4f64 on 16 x 16 blocks, tiles of 32 candidates (two
// 16-column MFMA tiles ct = 0, 1).  At MFMA step s (0..3) of block (I, J), A
// lane l holds Linv[16I + l%16][16J + 4s + l/16] and B lane l holds
// K*[16J + 4s + l/16][16ct + l%16]; K* is stored as (J, ct, s/2, lane)
// double2, component s%2.  Accumulator register r of lane l holds row
// l/16 + 4r, column l%16 of its tile (only column sums of squares are taken,
// so the row order does not matter here).  Same three phases and persistent
// loop as the fp32 kernel.
// ---------------------------------------------------------------------------
struct Post64 {
  int64_t n;
  int d, nb16;
  double scale[SCOOT_MAX_DIM];
  double c0, c1, c2;
  double s2, prior, ei_c;
  int warp;  // candidates through kumaraswamy(x, wa, wb) first
  double wa[SCOOT_MAX_DIM], wb[SCOOT_MAX_DIM];
  RowPlan16 plan;  // 16-row blocks
};

__device__ inline void load_block16(d2_t (&a)[2], const d2_t* ap, int k) {
  a[0] = ap[(size_t)(k * 2 + 0) * 64];
  a[1] = ap[(size_t)(k * 2 + 1) * 64];
}
// b[2 ct + s/2]
__device__ inline void load_b16(d2_t (&b)[4], const d2_t* ks, int J, int lane) {
#pragma unroll
  for (int ct = 0; ct < 2; ++ct)
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) b[2 * ct + s2] = ks[((J * 2 + ct) * 2 + s2) * 64 + lane];
}

// The 4 steps of a block on two chains (one per 16-candidate half), issued
// alternately; FIRST (the row's block J = 0) starts both from zero, so they need no
// clearing.
template <bool FIRST>
__device__ inline void mfma_block16(d4_t& l0, d4_t& l1, const d2_t (&a)[2], const d2_t (&b)[4]) {
  const d4_t zero = {0};
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bool z = FIRST && s2 == 0 && t == 0;
      l0 = __builtin_amdgcn_mfma_f64_16x16x4f64(a[s2][t], b[s2][t], z ? zero : l0, 0, 0, 0);
      l1 = __builtin_amdgcn_mfma_f64_16x16x4f64(a[s2][t], b[2 + s2][t], z ? zero : l1, 0, 0, 0);
    }
  }
}
__device__ inline void mfma_block16_at(int J, d4_t& l0, d4_t& l1, const d2_t (&a)[2], const d2_t (&b)[4]) {
  if (J == 0) mfma_block16<true>(l0, l1, a, b);
  else mfma_block16<false>(l0, l1, a, b);
}

// One tile's pass over the wave's blocks; the same schedule as wave_tile16f
// (one block of read-ahead, the A stream wrapping to the next tile).
__device__ inline void wave_tile16(const d2_t* __restrict__ ap, const d2_t* ks, uint64_t lo, uint64_t hi, int count,
                                   int lane, d2_t (&ax)[2], double& sq0, double& sq1) {
  d4_t l0 = __builtin_nondeterministic_value(l0), l1 = l0;
  constexpr uint64_t kMask = (1u << kRowBits16) - 1;
  int I = (int)(lo & kMask), J = 0;
  auto next_j = [&](int j, int i) { return j == i ? 0 : j + 1; };
  auto advance = [&]() {
    if (J == I) {
      double p0 = 0.0, p1 = 0.0;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        p0 = fma(l0[r], l0[r], p0);
        p1 = fma(l1[r], l1[r], p1);
      }
      sq0 += p0;
      sq1 += p1;
      J = 0;
      lo = (lo >> kRowBits16) | (hi << (64 - kRowBits16));
      hi >>= kRowBits16;
      I = (int)(lo & kMask);
    } else {
      ++J;
    }
  };
  d2_t ay[2], bx[4], by[4];
  load_b16(bx, ks, 0, lane);
  int k = 0;
  for (; k + 1 < count; k += 2) {
    load_block16(ay, ap, k + 1);
    load_b16(by, ks, next_j(J, I), lane);
    __builtin_amdgcn_sched_barrier(0);
    mfma_block16_at(J, l0, l1, ax, bx);
    __builtin_amdgcn_sched_barrier(0);
    advance();
    load_block16(ax, ap, k + 2 < count ? k + 2 : 0);
    load_b16(bx, ks, next_j(J, I), lane);
    __builtin_amdgcn_sched_barrier(0);
    mfma_block16_at(J, l0, l1, ay, by);
    __builtin_amdgcn_sched_barrier(0);
    advance();
  }
  if (k < count) {
    load_block16(ay, ap, 0);
    __builtin_amdgcn_sched_barrier(0);
    mfma_block16_at(J, l0, l1, ax, bx);
    __builtin_amdgcn_sched_barrier(0);
    advance();
    ax[0] = ay[0];
    ax[1] = ay[1];
  }
}

template <int WAVES, int D>
__global__ __launch_bounds__(WAVES * 64, 8 / WAVES) void posterior_f64_kernel(
    const float* __restrict__ Xc, const d2_t* __restrict__ linv, const double* __restrict__ xs,
    const double* __restrict__ alpha, double* __restrict__ mu_out, double* __restrict__ sd_out,
    double* __restrict__ ei_out, const Post64 a) {
  extern __shared__ __align__(16) unsigned char smem[];
  d2_t* ks = reinterpret_cast<d2_t*>(smem);  // [nb16][2 ct][2 s2][64] double2
  const int nb = a.nb16;
  double* sig_red = reinterpret_cast<double*>(ks + (size_t)nb * 2 * 2 * 64);  // [WAVES][4 g][32]
  double* mu_red = sig_red + WAVES * 4 * 32;                                   // [WAVES][2 h][32]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t n_tiles = (a.n + 31) >> 5;
  static_assert(WAVES % 2 == 0, "phase 1 relies on an even wave count");
  // 16-byte loads per observation row: the D coordinates and, below 16, alpha
  constexpr int kRowVec = D < kXsStride ? (D + 1 + 1) / 2 : kXsStride / 2;

  // plan entry of this wave, paired per SIMD as in the fp32 kernel
  int p = wave;
  if constexpr (WAVES == 8) {
    int* on_simd = reinterpret_cast<int*>(mu_red + WAVES * 2 * 32);  // [4]
    if (tid < 4) on_simd[tid] = 0;
    __syncthreads();
    const int simd = (int)((__builtin_amdgcn_s_getreg((31 << 11) | 4) >> 4) & 3);  // HW_ID.SIMD_ID
    int slot = 0;
    if (lane == 0) slot = atomicAdd(&on_simd[simd], 1);
    slot = __shfl(slot, 0);
    __syncthreads();
    if (on_simd[0] == 2 && on_simd[1] == 2 && on_simd[2] == 2 && on_simd[3] == 2) p = simd + 4 * slot;
    p = __builtin_amdgcn_readfirstlane(p);
  }
  const uint64_t rows_lo = a.plan.lo[p], rows_hi = a.plan.hi[p];
  const int count = a.plan.blk_start[p + 1] - a.plan.blk_start[p];
  const d2_t* ap = linv + (size_t)a.plan.blk_start[p] * 2 * 64 + lane;
  d2_t ax[2];
  if (count > 0) load_block16(ax, ap, 0);

  // lane -> candidate 32 tile + cl, row half h
  const int cl = lane & 31, h = lane >> 5;
  const int ct = cl >> 4, ncol = cl & 15;
  int64_t tile = blockIdx.x;
  float xr[D];
#pragma unroll
  for (int q = 0; q < D; ++q) xr[q] = Xc[min(tile * 32 + cl, a.n - 1) * D + q];

  for (; tile < n_tiles; tile += gridDim.x) {
    const int64_t c0 = tile * 32;
    double xc[D];
#pragma unroll
    for (int q = 0; q < D; ++q) {
      const double x = a.warp ? kumaraswamy((double)xr[q], a.wa[q], a.wb[q]) : (double)xr[q];
      xc[q] = x * a.scale[q];
    }
    const int64_t next = tile + gridDim.x;
    if (next < n_tiles) {
#pragma unroll
      for (int q = 0; q < D; ++q) xr[q] = Xc[min(next * 32 + cl, a.n - 1) * D + q];
    }

    __builtin_amdgcn_s_setprio(2);  // K* at a raised priority, as in the fp32 kernel
    // ---- phase 1: group G = 4J + 2 s2 + kk covers rows
    // 16J + 8 s2 + 4t + 2kk + h = 4G - 2kk + h + 4t (t = 0, 1) of block J;
    // WAVES is even, so kk = wave & 1 for all of a wave's groups and each
    // lane's rows advance by 4 WAVES per group.
    double mu_part = 0.0;
    const int ngroups = nb * 4;
    const int kw = wave & 1;
    const double* xg = xs + (size_t)(4 * wave - 2 * kw + h) * kXsStride;
    for (int G = wave; G < ngroups; G += WAVES, xg += 4 * WAVES * kXsStride) {
      const int J = G >> 2, s2 = (G >> 1) & 1;
      d2_t kv;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const double* xo = xg + 4 * t * kXsStride;
        double xv[kRowVec * 2];
#pragma unroll
        for (int r = 0; r < kRowVec; ++r) {
          const d2_t v2 = reinterpret_cast<const d2_t*>(xo)[r];
          xv[2 * r] = v2[0];
          xv[2 * r + 1] = v2[1];
        }
        double acc = 0.0;
#pragma unroll
        for (int q = 0; q < D; ++q) {
          const double df = xc[q] - xv[q];
          acc = fma(df, df, acc);
        }
        const double u = sqrt(acc);
        const double kval = fma(u, fma(u, a.c2, a.c1), a.c0) * exp2(-u);
        kv[t] = kval;
        const double al = D < kXsStride ? xv[D < kXsStride ? D : 0] : alpha[4 * G - 2 * kw + h + 4 * t];
        mu_part = fma(kval, al, mu_part);
      }
      ks[((J * 2 + ct) * 2 + s2) * 64 + (2 * kw + h) * 16 + ncol] = kv;
    }
    __syncthreads();

    __builtin_amdgcn_s_setprio(0);
    // ---- phase 2 ----------------------------------------------------------
    double sq0 = 0.0, sq1 = 0.0;
    if (count > 0) wave_tile16(ap, ks, rows_lo, rows_hi, count, lane, ax, sq0, sq1);

    // ---- phase 3: accumulator lane l holds column l % 16 of its tile ------
    const int g = lane >> 4;
    sig_red[(wave * 4 + g) * 32 + (lane & 15)] = sq0;
    sig_red[(wave * 4 + g) * 32 + 16 + (lane & 15)] = sq1;
    mu_red[(wave * 2 + h) * 32 + cl] = mu_part;
    __syncthreads();
    if (tid < 32) {
      const int64_t c = c0 + tid;
      if (c < a.n) {
        double ss = 0.0, mm = 0.0;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) {
#pragma unroll
          for (int gg = 0; gg < 4; ++gg) ss += sig_red[(w * 4 + gg) * 32 + tid];
          mm += mu_red[(w * 2 + 0) * 32 + tid] + mu_red[(w * 2 + 1) * 32 + tid];
        }
        const double sd = sqrt(fmax(a.s2 - ss, 0.0));
        const double mu = a.prior + mm;
        mu_out[c] = mu;
        sd_out[c] = sd;
        if (ei_out) ei_out[c] = partial_expectation_d(a.ei_c, mu, sd);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Input warping of the pool (fp32 path): every coordinate through
// w = 1 - (1 - x^a_k)^b_k, x clamped to [0, 1], in float and without
// cancellation: ln x from log1p(x - 1) above 1/2 (x - 1 exact there),
// 1 - x^a = -expm1(a ln x), w = -expm1(b ln(1 - x^a)).  Measured against
// double: 2e-7 absolute (forming x^a first and subtracting it from 1 loses
// up to 1.5e-4 near x = 1, where w is steep).  The fp64 path warps in double
// inside its kernel, by the same steps.
// ---------------------------------------------------------------------------
struct WarpArgs {
  float a[SCOOT_MAX_DIM], b[SCOOT_MAX_DIM];
};

__global__ __launch_bounds__(256) void warp_pool_kernel(const float* __restrict__ Xc, int64_t total, int d,
                                                        const WarpArgs w, float* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int k = (int)(i % d);
    const float x = fminf(fmaxf(Xc[i], 0.0f), 1.0f);
    const float lx = x > 0.5f ? log1pf(x - 1.0f) : logf(x);
    const float om = -expm1f(w.a[k] * lx);
    out[i] = -expm1f(w.b[k] * logf(om));
  }
}

int launch_warp_pool(const GPDevice& g, const float* Xc, int64_t n, float* out, void* stream) {
  const int64_t total = n * g.d;
  if (total == 0) return SCOOT_OK;
  WarpArgs w{};
  for (int k = 0; k < SCOOT_MAX_DIM; ++k) {
    w.a[k] = (float)g.warp_a[k];
    w.b[k] = (float)g.warp_b[k];
  }
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(warp_pool_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, Xc, total, g.d,
                     w, out);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("warp launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
namespace {

// Persistent grid: as many workgroups as the chip holds at once (each loops
// over tiles), at most one per tile.  0 when the workgroup does not fit.
int64_t persistent_grid(const void* kern, int threads, size_t lds, int64_t tiles) {
  int dev = 0, cus = 256, per_cu = 0;
  (void)hipGetDevice(&dev);
  (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, threads, lds) != hipSuccess || per_cu < 1)
    return 0;
  return std::min(tiles, (int64_t)cus * per_cu);
}

template <int WAVES, int D, bool KEEP_V>
int run32(const GPDevice& g, const float* Xc, int64_t n, float* mu, float* sd, float* ei, float* v_out,
          const Post32& a, hipStream_t s) {
  // K* tile, per-wave partial norms and means, four SIMD counters
  const size_t lds = (size_t)a.nb16 * 4 * 64 * 16 + 2 * WAVES * 64 * 4 + 16;
  auto kern = posterior_f32_kernel<WAVES, D, KEEP_V>;
  const int rc = allow_full_lds((const void*)kern, "posterior");
  if (rc != SCOOT_OK) return rc;
  const int64_t grid = persistent_grid((const void*)kern, WAVES * 64, lds, (n + 63) / 64);
  if (grid < 1) return fail(SCOOT_ERR_DEVICE, "posterior: workgroup does not fit on a compute unit");
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(WAVES * 64), lds, s, Xc,
                     (const f4_t*)g.linv, (const double*)g.xs, g.alpha32, mu, sd, ei, v_out, a);
  return SCOOT_OK;
}

template <int WAVES, int D>
int run64(const GPDevice& g, const float* Xc, int64_t n, double* mu, double* sd, double* ei,
          const Post64& a, hipStream_t s) {
  // K* tile, per-wave partial norms and means, four SIMD counters
  const int nb16 = g.m_pad / kBlk16;
  const size_t lds = (size_t)nb16 * 2 * 2 * 64 * 16 + WAVES * 4 * 32 * 8 + WAVES * 2 * 32 * 8 + 16;
  auto kern = posterior_f64_kernel<WAVES, D>;
  const int rc = allow_full_lds((const void*)kern, "posterior");
  if (rc != SCOOT_OK) return rc;
  const int64_t grid = persistent_grid((const void*)kern, WAVES * 64, lds, (n + 31) / 32);
  if (grid < 1) return fail(SCOOT_ERR_DEVICE, "posterior: workgroup does not fit on a compute unit");
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(WAVES * 64), lds, s, Xc,
                     (const d2_t*)g.linv, (const double*)g.xs, g.alpha, mu, sd, ei, a);
  return SCOOT_OK;
}

template <int D, typename F>
int by_d_rec(int d, F&& f) {
  if constexpr (D > SCOOT_MAX_DIM) {
    return fail(SCOOT_ERR_UNSUPPORTED, "posterior: d exceeds SCOOT_MAX_DIM");
  } else {
    if (d == D) return f(std::integral_constant<int, D>());
    return by_d_rec<D + 1>(d, std::forward<F>(f));
  }
}

}  // namespace

int launch_posterior(const GPDevice& g, const float* Xc, int64_t n, void* mu, void* sigma,
                     const double* ei_c, void* ei, void* stream, float* v_out, bool xc_warped, int64_t v_ld) {
  if (n == 0) return SCOOT_OK;
  if (n >= ((int64_t)1 << 37)) return fail(SCOOT_ERR_UNSUPPORTED, "posterior: n too large");
  hipStream_t s = (hipStream_t)stream;
  int rc;
  if (g.dt == SCOOT_F32 && g.warp && !xc_warped) {
    float* Xw = (float*)device_scratch((size_t)n * g.d * sizeof(float), 5);
    if (!Xw) return fail(SCOOT_ERR_NO_MEMORY, "posterior: warped pool allocation failed");
    rc = launch_warp_pool(g, Xc, n, Xw, stream);
    if (rc != SCOOT_OK) return rc;
    Xc = Xw;
  }
  if (g.dt == SCOOT_F32) {
    Post32 a{};
    a.n = n;
    a.d = g.d;
    a.nb16 = g.m_pad / kBlk16;
    for (int k = 0; k < SCOOT_MAX_DIM; ++k) a.scale[k] = g.scale64[k];
    a.c0 = g.coef32[0];
    a.c1 = g.coef32[1];
    a.c2 = g.coef32[2];
    a.s2 = g.s2;
    a.prior = g.c;
    a.ei_c = ei_c ? *ei_c : 0.0;
    a.plan = plan_rows16(a.nb16, posterior_waves(g.nb));
    a.v_ld = v_ld > 0 ? v_ld : n;
    for (int e = 0; e < 8; ++e)
      if (a.plan.nrows[e] > kMaxRows16) return fail(SCOOT_ERR_UNSUPPORTED, "posterior: row plan does not pack");
    float* e = ei_c ? (float*)ei : nullptr;
    rc = by_d_rec<1>(g.d, [&](auto Dc) {
      constexpr int D = decltype(Dc)::value;
      float *m32 = (float*)mu, *s32 = (float*)sigma;
      if (posterior_waves(g.nb) == 8)
        return v_out ? run32<8, D, true>(g, Xc, n, m32, s32, e, v_out, a, s)
                     : run32<8, D, false>(g, Xc, n, m32, s32, e, nullptr, a, s);
      return v_out ? run32<4, D, true>(g, Xc, n, m32, s32, e, v_out, a, s)
                   : run32<4, D, false>(g, Xc, n, m32, s32, e, nullptr, a, s);
    });
  } else {
    Post64 a{};
    a.n = n;
    a.d = g.d;
    a.warp = g.warp && !xc_warped ? 1 : 0;
    for (int k = 0; k < SCOOT_MAX_DIM; ++k) {
      a.wa[k] = g.warp_a[k];
      a.wb[k] = g.warp_b[k];
    }
    a.nb16 = g.m_pad / kBlk16;
    a.plan = plan_rows16(a.nb16, posterior_waves(g.nb));
    for (int e = 0; e < 8; ++e)
      if (a.plan.nrows[e] > kMaxRows16) return fail(SCOOT_ERR_UNSUPPORTED, "posterior: row plan does not pack");
    for (int k = 0; k < SCOOT_MAX_DIM; ++k) a.scale[k] = g.scale64[k];
    a.c0 = g.coef64[0];
    a.c1 = g.coef64[1];
    a.c2 = g.coef64[2];
    a.s2 = g.s2;
    a.prior = g.c;
    a.ei_c = ei_c ? *ei_c : 0.0;
    double* e = ei_c ? (double*)ei : nullptr;
    rc = by_d_rec<1>(g.d, [&](auto Dc) {
      constexpr int D = decltype(Dc)::value;
      double *m64 = (double*)mu, *s64 = (double*)sigma;
      if (posterior_waves(g.nb) == 8) return run64<8, D>(g, Xc, n, m64, s64, e, a, s);
      return run64<4, D>(g, Xc, n, m64, s64, e, a, s);
    });
  }
  if (rc != SCOOT_OK) return rc;
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("posterior launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}

}  // namespace scoot
