// The GP's negative log likelihood and its gradient in the hyperparameters,
// evaluated on the device in fp64 (Sec. 4.3: the noise level and the other
// hyperparameters are learned by maximum likelihood).  The search itself (the
// box-constrained L-BFGS of host_mle.cpp) stays on the host and calls this
// once per trial point.
//
// With r = y - c, K = k_theta(X, X) + tau2 I (m x m), K = L L^T, u = L^-1 r and
// W = alpha alpha^T - K^-1:
//   NLL = 1/2 u^T u + 1/2 log det K + m/2 log(2 pi),   alpha = K^-1 r = L^-T u
//   dNLL/dtheta_p = -1/2 sum_ij W_ij (dK/dtheta_p)_ij
// with the derivatives of the covariance written out in host_mle.cpp.
//
// Matrices are 16 x 16 blocks, m padded to a multiple of 16 with identity rows
// (their covariance with real rows is 0, their diagonal 1, their r 0: log det,
// the quadratic form and the gradient do not see them).  The kernels of one
// evaluation, on one stream:
//   W. (warp learned) the warped inputs and their derivatives;
//   K. K, one 16 x 16 block per workgroup;
//   A. one workgroup (8 waves): the Cholesky factor L by 16-column block
//      steps: the diagonal block factored and inverted by one wave in
//      registers (a rank-1 update per column on v_mfma_f64_16x16x4f64), the
//      panel below it as the product with that inverse and the trailing
//      update, both on the matrix cores, and u = L^-1 r by forward
//      substitution alongside; the next diagonal block is factored as soon
//      as it is updated, by a wave whose SIMD the others leave free;
// and, when the gradient is wanted,
//   T. L^-1 and alpha = L^-T u, one block column per workgroup (the columns
//      are independent);
//   B. the gradient, one lower block per workgroup: the block of
//      K^-1 = L^-T L^-1 on the matrix cores, then one element of W per
//      thread, the covariance and its derivatives recomputed, partial sums
//      per workgroup.
// The kernels write their results (status, pivot products, |u|^2 per block,
// partial gradient sums) straight into pinned host memory, and the host adds
// them.  Every operation is in double and every sum has a fixed order, so an
// evaluation is deterministic.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <utility>
#include <vector>

#include "internal.h"

namespace scoot {
namespace {

typedef double d2_t __attribute__((ext_vector_type(2)));
typedef double d4_t __attribute__((ext_vector_type(4)));

constexpr int kNllWaves = 8;
constexpr int kNllThreads = kNllWaves * 64;
constexpr int kMaxTheta = 3 * SCOOT_MAX_DIM + 2;
constexpr int kGradThreads = 256;
constexpr int kGradWaves = kGradThreads / 64;
constexpr double kRoot5 = 2.23606797749978969641;
constexpr double kRoot3 = 1.73205080756887729353;
constexpr double kLog2PiD = 1.83787706640934548356;

struct NllArgs {
  const double* X;  // m x d inputs as the covariance sees them (raw when the warp is learned)
  const double* r;  // m_pad: y - c, 0 beyond m
  double* L;        // nb x nb blocks: K, then its lower factor (blocks I >= J)
  double* Xi;       // nb x nb blocks: L^-1 (blocks I >= J)
  double* Di;       // nb blocks: inverses of L's diagonal blocks
  double* Xw;       // m x d warped inputs (warp learned)
  double* Ga;       // m x d: d w / d log a (warp learned)
  double* Gb;       // m x d: d w / d log b (warp learned)
  double* alpha;    // m_pad: K^-1 r
  double* u;        // m_pad: L^-1 r
  double* out;      // [1] 1 when K is numerically positive definite, 0 when not, 2 when a wait ran out
  // Pinned host memory the kernels write their results to: [0] the status of
  // out[1], [1 .. nb] the product of each diagonal block's pivots (real rows),
  // [nb + 1 ..] u (16 nb values), then nb (nb + 1) / 2 x P partial gradient
  // sums (one row per lower block); the host adds them in a fixed order.
  double* hout;
  int m, nb, d, m52, learn_warp;
  double theta[kMaxTheta];
};

// ---- 16 x 16 blocks on the fp64 matrix cores -------------------------------
// v_mfma_f64_16x16x4f64 takes, in lane l (g = l / 16, c = l % 16), A[c][g] and
// B[g][c] of a 16 x 4 by 4 x 16 product and accumulates into a block whose
// register r of lane l is row g + 4r, column c ("C layout").  A 16-deep
// product is four such steps s, with a[s] = A[c][4s + g], b[s] = B[4s + g][c].
__device__ inline d4_t mma16(d4_t acc, const double (&a)[4], const double (&b)[4]) {
#pragma unroll
  for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a[s], b[s], acc, 0, 0, 0);
  return acc;
}
__device__ inline d4_t zero4() { return d4_t{0.0, 0.0, 0.0, 0.0}; }
// C layout of a row-major block in memory: element 64 r + l.
__device__ inline d4_t ld_c(const double* blk, int lane) {
  return d4_t{blk[lane], blk[64 + lane], blk[128 + lane], blk[192 + lane]};
}
__device__ inline void st_c(double* blk, const d4_t& v, int lane) {
#pragma unroll
  for (int r = 0; r < 4; ++r) blk[64 * r + lane] = v[r];
}
// M[c][4s + g] of a row-major block (A operand from M, B operand from M^T)
__device__ inline void ld_rows(const double* blk, int lane, double (&a)[4]) {
  const double* p = blk + (lane & 15) * 16 + (lane >> 4);
#pragma unroll
  for (int s = 0; s < 4; ++s) a[s] = p[4 * s];
}
// M[4s + g][c] of a row-major block (B operand from M, A operand from M^T): the C layout
__device__ inline void ld_cols(const double* blk, int lane, double (&a)[4]) {
#pragma unroll
  for (int s = 0; s < 4; ++s) a[s] = blk[64 * s + lane];
}
// LDS slots of 256 doubles laid out so that a lane's four operand values are
// contiguous at 4 l: "row slots" hold M[c][4s + g], "column slots" M[4s + g][c].
__device__ inline void ld_slot(const double* slot, int lane, double (&a)[4]) {
  const d2_t* p = reinterpret_cast<const d2_t*>(slot + 4 * lane);
  const d2_t x = p[0], y = p[1];
  a[0] = x[0], a[1] = x[1], a[2] = y[0], a[3] = y[1];
}
// a block in C layout into a column slot (position 4 l + r)
__device__ inline void st_col_slot(double* slot, const d4_t& v, int lane) {
  d2_t* p = reinterpret_cast<d2_t*>(slot + 4 * lane);
  p[0] = d2_t{v[0], v[1]};
  p[1] = d2_t{v[2], v[3]};
}
// position of element (row, col) in a row slot
__device__ inline int row_slot_pos(int row, int col) { return ((col & 3) * 16 + row) * 4 + (col >> 2); }
__device__ inline void st_row_slot(double* slot, const d4_t& v, int lane) {
  const int g = lane >> 4, c = lane & 15;
#pragma unroll
  for (int r = 0; r < 4; ++r) slot[row_slot_pos(g + 4 * r, c)] = v[r];
}

// Next (I, J), J <= I, of a lower triangle enumerated row by row, n steps on.
__device__ inline void advance_lower(int& I, int& J, int n) {
  J += n;
  while (J > I) {
    J -= I + 1;
    ++I;
  }
}

// Lanes of one wave exchanging values through LDS: every LDS access issued
// before has completed (s_waitcnt lgkmcnt(0)) and the compiler moves no memory
// access across.
__device__ inline void wave_lds_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

// Workgroup barrier for waves that exchange data through LDS only: their LDS
// accesses have completed, their global stores may still be in flight.
__device__ inline void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Order-fixed sum over the 64 lanes.
__device__ inline double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// The warp of x and its derivatives in log a and log b (0 at x = 0 and 1),
// without cancellation: ln x from log1p(x - 1) above 1/2, 1 - x^a = -expm1(a ln x).
__device__ inline void warp_derivatives(double x, double a, double b, double* w, double* ga, double* gb) {
  x = x < 0.0 ? 0.0 : (x > 1.0 ? 1.0 : x);
  *w = kumaraswamy(x, a, b);
  if (x <= 0.0 || x >= 1.0) {
    *ga = *gb = 0.0;
    return;
  }
  const double lx = x > 0.5 ? log1p(x - 1.0) : log(x);
  const double u = exp(a * lx);
  const double l1u = log(-expm1(a * lx));  // ln(1 - x^a)
  *ga = a * b * exp((b - 1.0) * l1u) * u * lx;
  *gb = -b * exp(b * l1u) * l1u;
}

// Matern covariance at scaled distance t = sqrt(2 nu) r (without tau2).
__device__ inline double matern(bool m52, double s2, double t, double e) {
  return m52 ? s2 * (1.0 + t + t * t / 3.0) * e : s2 * (1.0 + t) * e;
}

// ---- kernel W: warped inputs and their derivatives (warp learned) ---------
__global__ __launch_bounds__(256) void nll_warp_kernel(NllArgs a) {
  const int d = a.d, idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= a.m * d) return;
  const int k = idx % d;
  warp_derivatives(a.X[idx], exp(a.theta[d + 2 + k]), exp(a.theta[2 * d + 2 + k]), &a.Xw[idx], &a.Ga[idx],
                   &a.Gb[idx]);
}

// ---- kernel K: the covariance, one lower 16 x 16 block per workgroup --------
// Diagonal blocks in full; padding rows and columns are those of the identity.
// Each block is written transposed (column-major), the layout kernel A reads.
__global__ __launch_bounds__(256) void nll_cov_kernel(NllArgs a) {
  __shared__ double sXi[16 * SCOOT_MAX_DIM], sXj[16 * SCOOT_MAX_DIM], sIl[SCOOT_MAX_DIM];
  const int nb = a.nb, m = a.m, d = a.d, t = threadIdx.x;
  int I = 0, J = 0;
  advance_lower(I, J, blockIdx.x);
  const bool m52 = a.m52 != 0;
  const double s2 = exp(a.theta[d]), tau2 = exp(a.theta[d + 1]);
  const double root = m52 ? kRoot5 : kRoot3;
  const double* X = a.learn_warp ? a.Xw : a.X;
  if (t < 16 * d) {
    const int r = t / d, k = t % d, i = 16 * I + r, j = 16 * J + r;
    sXi[t] = i < m ? X[(size_t)i * d + k] : 0.0;
    sXj[t] = j < m ? X[(size_t)j * d + k] : 0.0;
  }
  if (t < d) sIl[t] = exp(-a.theta[t]);
  __syncthreads();
  // block (I, J) is stored transposed: thread t holds element (ii, jj) at t = 16 jj + ii
  const int jj = t >> 4, ii = t & 15, i = 16 * I + ii, j = 16 * J + jj;
  double v;
  if (i < m && j < m) {
    double r2 = 0.0;
    for (int k = 0; k < d; ++k) {
      const double q = (sXi[ii * d + k] - sXj[jj * d + k]) * sIl[k];
      r2 += q * q;
    }
    const double tt = root * sqrt(r2);
    v = matern(m52, s2, tt, exp(-tt)) + (i == j ? tau2 : 0.0);
  } else {
    v = i == j ? 1.0 : 0.0;
  }
  a.L[((size_t)I * nb + J) * 256 + t] = v;
}

// The 64-bit value v of lane src, to every lane (as a scalar).
__device__ inline double lane_bcast(double v, int src) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(v);
  const int lo = __builtin_amdgcn_readlane((int)(unsigned)b, src);
  const int hi = __builtin_amdgcn_readlane((int)(unsigned)(b >> 32), src);
  return __hiloint2double(hi, lo);
}

// Factors the 16 x 16 diagonal block kk, held in C layout by one wave, and
// inverts the factor on the way.  Column c: the pivot p = D[c][c] comes from
// one lane; l = D[c][.] / sqrt(p) (row c, by symmetry column c of L) sits in
// register c / 4 of row group c % 4, which is where v_mfma_f64_16x16x4f64 takes
// both operands of its k = c % 4 slice, so one MFMA subtracts l l^T from the
// whole block.  The same l against row c of Y (Y = I at the start) scaled by
// 1 / L[c][c], which is row c of L^-1, carries out the forward substitution of
// L Y = I a column at a time.  Stores L_kk column-major to memory, L_kk^-1
// row-major to memory (Di) and as a row slot (sX), the product of the pivots of
// real rows to sProd[kk]; raises sFlag[0] when such a pivot is not above floor
// (or a padding pivot is not positive).
__device__ inline void diag_factor(const NllArgs& a, int kk, d4_t D, double* sX, double* sProd, int* sFlag,
                                   double floor, int lane) {
  const int g = lane >> 4, j = lane & 15, real = min(16, a.m - 16 * kk);
  d4_t Lt = zero4(), X = zero4(), Y;  // Lt: L^T in C layout (row c of Lt = column c of L)
#pragma unroll
  for (int r = 0; r < 4; ++r) Y[r] = g + 4 * r == j ? 1.0 : 0.0;
  double prod = 1.0;
  bool bad = false;
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    const int cg = c & 3, cr = c >> 2;
    const double piv = lane_bcast(D[cr], cg * 16 + c);
    const bool real_row = c < real;
    bad = bad || !(piv > (real_row ? floor : 0.0));
    prod *= real_row ? piv : 1.0;
    // 1 / sqrt(piv): the hardware estimate and two Newton steps (each about
    // squares the relative error), a shorter dependent chain than sqrt and
    // a division
    double ic = __builtin_amdgcn_rsq(piv);
    const double h = 0.5 * piv;
    ic = ic * fma(-h * ic, ic, 1.5);
    ic = ic * fma(-h * ic, ic, 1.5);
    const bool mine = g == cg;
    const double l = mine && j >= c ? D[cr] * ic : 0.0;  // L[j][c], 0 above the diagonal
    const double y = mine ? Y[cr] * ic : 0.0;            // (L^-1)[c][j]
    if (mine) {
      Lt[cr] = l;
      X[cr] = y;
    }
    D = __builtin_amdgcn_mfma_f64_16x16x4f64(-l, l, D, 0, 0, 0);
    Y = __builtin_amdgcn_mfma_f64_16x16x4f64(-l, y, Y, 0, 0, 0);
  }
  st_c(a.L + ((size_t)kk * a.nb + kk) * 256, Lt, lane);  // L_kk column-major
  st_c(a.Di + (size_t)kk * 256, X, lane);
  st_row_slot(sX, X, lane);
  if (lane == 0) {
    sProd[kk] = prod;
    if (bad) sFlag[0] = 1;
  }
}

// Forward substitution for u = L^-1 r, the diagonal block's part: u_kk =
// L_kk^-1 r_kk with L_kk^-1 from its row slot sX and r_kk (the residual) from
// LDS, as one product C = R L_kk^-T where every row of R is r_kk, so that
// every row of C is u_kk; to sU (16), to memory and to the host.
__device__ inline void diag_solve(const NllArgs& a, int kk, const double* sX, const double* rk, double* sU,
                                  int lane) {
  const int g = lane >> 4, c = lane & 15;
  double av[4], bv[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) av[s] = rk[4 * s + g];
  ld_slot(sX, lane, bv);  // (L_kk^-1)^T as a B operand
  const d4_t v = mma16(zero4(), av, bv);
  if (lane < 16) {
    sU[c] = v[0];
    a.u[16 * kk + c] = v[0];
    a.hout[1 + a.nb + 16 * kk + c] = v[0];
  }
}

// The residual's update by a panel block: r_i -= L_ik u_k, with L_ik from its
// row slot (lane (g, c) holds L_ik[c][4s + g]) and u_k in LDS.
__device__ inline void resid_update(double* ri, const double* slot, const double* uk, int lane) {
  const int g = lane >> 4;
  double lv[4];
  ld_slot(slot, lane, lv);
  double s = lv[0] * uk[g] + lv[1] * uk[4 + g] + lv[2] * uk[8 + g] + lv[3] * uk[12 + g];
  s += __shfl_xor(s, 16);
  s += __shfl_xor(s, 32);
  if (lane < 16) ri[lane] -= s;
}

// ---- kernel A: the Cholesky factor L and the inverses of its diagonal blocks --
// Blocks are held transposed: the covariance kernel writes block (I, J)
// column-major, the workers' registers hold A_ij^T in C layout (A_ij as an A
// operand), and the factor goes to memory column-major too.  The worker blocks, (i, j) with 1 <= j <= i
// but (1, 1), are listed by decreasing j (then increasing i) and dealt round
// robin to the workers; at step k a worker's blocks with j >= k + 1 form a
// prefix of its share, so each step's work is balanced and the first kRes
// blocks of a share, the longest-lived, stay in registers for the whole
// factorization (the others go through memory each step).
constexpr int kRes = 8;

__global__ __launch_bounds__(kNllThreads) void nll_factor_kernel(NllArgs a) {
  extern __shared__ __align__(16) double sm[];
  const int nb = a.nb, d = a.d;
  double* sPan = sm;                          // 2 x nb row slots: the panels of columns k and k + 1
  double* sX = sPan + (size_t)2 * nb * 256;   // row slot: the inverse of the newest diagonal factor
  double* sDiag = sX + 256;                   // 2 x 256: the next diagonal blocks as updated (C layout)
  double* sProd = sDiag + 512;                // per diagonal block: product of its pivots
  double* sR = sProd + SCOOT_MAX_OBS / 16;    // nb x 16: r, then the forward substitution's residual
  double* sU = sR + (size_t)nb * 16;          // 2 x 16: u_k, by k % 2
  // [0] a pivot not above its floor, [1] the last diagonal block factored,
  // [2] a wait for it ran out
  int* sFlag = reinterpret_cast<int*>(sU + 32);
  int* sSimd = sFlag + 4;                     // kNllWaves: the SIMD each wave runs on
  int* sList = sSimd + kNllWaves;             // the worker blocks, (i << 8) | j

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if (lane == 0) sSimd[wave] = (int)((__builtin_amdgcn_s_getreg((31 << 11) | 4) >> 4) & 3);  // HW_ID.SIMD_ID
  if (tid < 4) sFlag[tid] = 0;
  for (int i = tid; i < nb * 16; i += kNllThreads) sR[i] = a.r[i];
  const int n_list = nb > 1 ? nb * (nb - 1) / 2 - 1 : 0;
  for (int n = tid; n < n_list; n += kNllThreads) {
    int start = 0;
    for (int j = nb - 1; j >= 1; --j) {
      const int lo = j == 1 ? 2 : j, cnt = nb - lo;
      if (n < start + cnt) {
        sList[n] = ((lo + n - start) << 8) | j;
        break;
      }
      start += cnt;
    }
  }
  const double s2 = exp(a.theta[d]), tau2 = exp(a.theta[d + 1]);
  // A pivot that is not above 1e-13 of its original diagonal entry (s2 + tau2)
  // means K is not numerically positive definite (the host factor's rule).
  const double floor = 1e-13 * (s2 + tau2);
  lds_barrier();
  // The trailing update goes to the waves that do not share wave 0's SIMD:
  // its vector ALU and the matrix unit are one datapath, so a neighbour's
  // matrix instructions would stall the factorization.
  int worker = -1, W = 0;
  for (int w = 1; w < kNllWaves; ++w)
    if (sSimd[w] != sSimd[0]) {
      if (w == wave) worker = W;
      ++W;
    }
  if (W == 0) {  // every wave on one SIMD: all but wave 0 work
    worker = wave - 1;
    W = kNllWaves - 1;
  }
  // a worker's blocks among the first S of the list; the blocks with j >= c
  // are the first (nb - c)(nb - c + 1) / 2 (less (1, 1) when c = 1)
  auto mine_below = [&](int S) { return S > worker ? (S - 1 - worker) / W + 1 : 0; };
  auto from_col = [&](int c) { return (nb - c) * (nb - c + 1) / 2 - (c <= 1 ? 1 : 0); };

  // ---- Cholesky factor, 16 columns per step --------------------------------
  // Before step k the panel of column k, L_ik (i > k), is in row slots and
  // L_kk^-1 in sX.  Step k: wave 0 updates block (k+1, k+1), factors and
  // inverts it; the workers apply column k to their blocks with j >= k+1,
  // A_ij^T -= L_jk L_ik^T (block (k+2, k+2) also to wave 0 through LDS), and
  // once wave 0 has published the new inverse turn their blocks of column
  // k+1 into the panel, L_i,k+1^T = L_k+1,k+1^-1 A_i,k+1^T.  The waves share
  // data through LDS only (a worker reads back only blocks it wrote), so the
  // one barrier per step does not wait for global stores.
  constexpr int kCol0 = (SCOOT_MAX_OBS / 16 - 1 + kNllWaves - 2) / (kNllWaves - 1);  // column-0 blocks per wave
  double c0[kCol0][4];
  d4_t res[kRes];  // a worker's first kRes blocks (transposed, C layout)
  int rij[kRes];
  const int n_share = worker >= 0 ? mine_below(n_list) : 0;
#pragma unroll
  for (int s = 0; s < kRes; ++s) rij[s] = s < n_share ? __builtin_amdgcn_readfirstlane(sList[worker + W * s]) : 0;
  if (wave == 0) {
    diag_factor(a, 0, ld_c(a.L, lane), sX, sProd, sFlag, floor, lane);
    wave_lds_sync();
    diag_solve(a, 0, sX, sR, sU, lane);
  } else {
    // the blocks of column 0, while wave 0 factors block (0, 0)
#pragma unroll
    for (int t = 0; t < kCol0; ++t) {
      const int i = wave + (kNllWaves - 1) * t;
      if (i < nb) ld_cols(a.L + (size_t)i * nb * 256, lane, c0[t]);  // A_i0^T as a B operand
    }
  }
  lds_barrier();
  // the panel of column 0: L_i0^T = L_00^-1 A_i0^T (C layout, so column-major
  // to memory and a row slot of L_i0 as it stands)
  if (wave != 0) {
    double xv[4];
    ld_slot(sX, lane, xv);
#pragma unroll
    for (int t = 0; t < kCol0; ++t) {
      const int i = wave + (kNllWaves - 1) * t;
      if (i < nb) {
        const d4_t v = mma16(zero4(), xv, c0[t]);
        st_c(a.L + (size_t)i * nb * 256, v, lane);
        st_col_slot(sPan + (size_t)i * 256, v, lane);
      }
    }
    // the worker's resident blocks
#pragma unroll
    for (int s = 0; s < kRes; ++s)
      if (s < n_share) res[s] = ld_c(a.L + ((size_t)(rij[s] >> 8) * nb + (rij[s] & 255)) * 256, lane);
  }
  lds_barrier();
  int cur = 0;
  for (int k = 0; k + 1 < nb; ++k, cur ^= 1) {
    if (sFlag[0] || sFlag[2]) break;
    const double* pc = sPan + (size_t)cur * nb * 256;  // panel of column k
    double* pn = sPan + (size_t)(cur ^ 1) * nb * 256;  // panel of column k + 1, being made
    if (wave == 0) {
      const int i = k + 1;
      // block (k+1, k+1) as the previous step's update left it (from its
      // worker through LDS, buffer k % 2; at k = 0 the covariance itself)
      const double* dg = sDiag + (k & 1) * 256;
      d4_t acc = k == 0 ? ld_c(a.L + ((size_t)i * nb + i) * 256, lane)
                        : d4_t{dg[lane], dg[64 + lane], dg[128 + lane], dg[192 + lane]};
      double av[4], bv[4];
      ld_slot(pc + (size_t)i * 256, lane, bv);
#pragma unroll
      for (int s = 0; s < 4; ++s) av[s] = -bv[s];
      acc = mma16(acc, av, bv);
      diag_factor(a, i, acc, sX, sProd, sFlag, floor, lane);
      wave_lds_sync();  // the inverse is in LDS
      if (lane == 0) __hip_atomic_store(&sFlag[1], i, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
      // while the workers make the panel: the residual of block k+1 takes
      // column k's last term (the other blocks' come from the workers this
      // step), then u_k+1
      resid_update(sR + 16 * i, pc + (size_t)i * 256, sU + (k & 1) * 16, lane);
      diag_solve(a, i, sX, sR + 16 * i, sU + (i & 1) * 16, lane);
    } else if (worker >= 0) {
      const int n_trail = mine_below(from_col(k + 2));  // the share's blocks with j >= k+2
      const int n_act = mine_below(from_col(k + 1));    // ... with j >= k+1
      double* sNext = sDiag + ((k + 1) & 1) * 256;
      // the inverse of block (k+1, k+1) from wave 0 (a bounded wait)
      bool have_x = false;
      double xv[4];
      auto wait_x = [&]() {
        if (have_x) return;
        for (int spins = 0; __hip_atomic_load(&sFlag[1], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < k + 1;) {
          if (++spins > (1 << 22)) {
            if (lane == 0) sFlag[2] = 1;
            break;
          }
          __builtin_amdgcn_s_sleep(2);
        }
        wave_lds_sync();
        ld_slot(sX, lane, xv);
        have_x = true;
      };
      // resident blocks: the update
#pragma unroll
      for (int s = 0; s < kRes; ++s) {
        const int i = rij[s] >> 8, j = rij[s] & 255;
        if (s < n_act && !(i == k + 1 && j == k + 1)) {
          double av[4], bv[4];
          ld_slot(pc + (size_t)j * 256, lane, av);
          ld_slot(pc + (size_t)i * 256, lane, bv);
#pragma unroll
          for (int q = 0; q < 4; ++q) av[q] = -av[q];
          res[s] = mma16(res[s], av, bv);
          if (i == k + 2 && j == k + 2) st_c(sNext, res[s], lane);
        }
        __builtin_amdgcn_sched_barrier(0);  // a block's operands loaded where it is updated
      }
      // column k's term of the forward substitution for the blocks below k+1,
      // r_i -= L_ik u_k, round robin over the workers
      for (int i = k + 2 + worker; i < nb; i += W) resid_update(sR + 16 * i, pc + (size_t)i * 256, sU + (k & 1) * 16, lane);
      // the others, four at a time, their loads first: the blocks with
      // j >= k+2 back to memory, then those of column k+1 into the panel
      for (int e0 = kRes; e0 < n_act; e0 += 4) {
        d4_t acc[4];
        int ij[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          ij[u] = __builtin_amdgcn_readfirstlane(sList[worker + W * (e0 + u < n_act ? e0 + u : e0)]);
          acc[u] = ld_c(a.L + ((size_t)(ij[u] >> 8) * nb + (ij[u] & 255)) * 256, lane);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int i = ij[u] >> 8, j = ij[u] & 255;
          if (e0 + u < n_act && !(i == k + 1 && j == k + 1)) {
            double av[4], bv[4];
            ld_slot(pc + (size_t)j * 256, lane, av);
            ld_slot(pc + (size_t)i * 256, lane, bv);
#pragma unroll
            for (int q = 0; q < 4; ++q) av[q] = -av[q];
            acc[u] = mma16(acc[u], av, bv);
            if (e0 + u < n_trail) {
              st_c(a.L + ((size_t)i * nb + j) * 256, acc[u], lane);
              if (i == k + 2 && j == k + 2) st_c(sNext, acc[u], lane);
            }
          }
        }
        if (e0 + 3 >= n_trail) {  // a block of column k+1 among the four
          wait_x();
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int i = ij[u] >> 8;
            if (e0 + u >= n_trail && e0 + u < n_act && i != k + 1) {
              const double tv[4] = {acc[u][0], acc[u][1], acc[u][2], acc[u][3]};
              const d4_t v = mma16(zero4(), xv, tv);
              st_c(a.L + ((size_t)i * nb + k + 1) * 256, v, lane);
              st_col_slot(pn + (size_t)i * 256, v, lane);
            }
          }
        }
      }
      // resident blocks of column k+1: the panel
      if (n_trail < kRes && n_trail < n_act) {
        wait_x();
#pragma unroll
        for (int s = 0; s < kRes; ++s) {
          const int i = rij[s] >> 8;
          if (s >= n_trail && s < n_act && i != k + 1) {
            const double tv[4] = {res[s][0], res[s][1], res[s][2], res[s][3]};
            const d4_t v = mma16(zero4(), xv, tv);
            st_c(a.L + ((size_t)i * nb + k + 1) * 256, v, lane);
            st_col_slot(pn + (size_t)i * 256, v, lane);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    lds_barrier();
  }
  // status: 1 factored, 0 not positive definite, 2 a wait ran out (reported as
  // a device failure)
  const double status = sFlag[2] ? 2.0 : (sFlag[0] ? 0.0 : 1.0);
  if (tid == 0) {
    a.out[1] = status;
    a.hout[0] = status;
  }
  if (status == 1.0 && tid < nb) a.hout[1 + tid] = sProd[tid];
}

// ---- kernel T: L^-1, one block column per workgroup ---------------------------
// Column j: X_jj = Di_j, and for i > j
//   X_ij = -Di_i S_ij,   S_ij = sum_{k=j}^{i-1} L_ik X_kj.
// Right-looking: as soon as X_kj is known every later row i adds its term
// L_ik X_kj to S_ij, which the wave that finishes row i keeps in registers
// (rows dealt round robin to the waves, R per wave at most); the owner of row
// k+1 then finishes X_k+1,j into LDS, where the column stays until it is
// written out at the end.  L was written by another compute unit, so its
// blocks (column-major: an A operand is a contiguous read) are loaded
// kTriAhead steps ahead into a ring of registers, and Di up front; every step
// issues the same loads (a row with nothing to load reads block (0, 0)), so
// each wait is for exactly the load it needs.
constexpr int kTriWaves = 8;
constexpr int kTriMaxRows = (SCOOT_MAX_OBS / 16 - 1 + kTriWaves - 1) / kTriWaves;
constexpr int kTriAhead = 3;

template <int R>
struct TriState {
  d4_t S[R];
  double Lv[kTriAhead][R][4];  // ring: L_ik for steps k, k+1, k+2 in slot (k - j) % 3
  double Dv[R][4];             // Di_i
};

// Step k of column j; ring slot B holds L_ik.  Steps past the column's end
// only load and wait, so that every wave runs the same number of barriers.
template <int R, int B>
__device__ inline void tri_step(const NllArgs& a, TriState<R>& st, double* sXcol, int j, int k, int wave,
                                int lane) {
  const int nb = a.nb;
  double xv[4];
  ld_slot(sXcol + (size_t)(k < nb ? k : nb - 1) * 256, lane, xv);  // X_kj as a B operand
#pragma unroll
  for (int t = 0; t < R; ++t) {
    const int i = j + 1 + wave + kTriWaves * t;
    if (i > k && i < nb) {  // row k+1 (if this wave's) comes first
      st.S[t] = mma16(st.S[t], st.Lv[B][t], xv);
      if (i == k + 1) {
        double nd[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) nd[s] = -st.Dv[t][s];
        const double sv[4] = {st.S[t][0], st.S[t][1], st.S[t][2], st.S[t][3]};  // S as a B operand is its own C layout
        st_col_slot(sXcol + (size_t)i * 256, mma16(zero4(), nd, sv), lane);
      }
    }
    const bool next = i < nb && k + kTriAhead < i;
    ld_cols(a.L + (next ? ((size_t)i * nb + k + kTriAhead) * 256 : 0), lane, st.Lv[B][t]);
  }
  lds_barrier();
}

template <int R>
__global__ __launch_bounds__(kTriWaves * 64) void nll_trtri_kernel(NllArgs a) {
  extern __shared__ __align__(16) double sXcol[];  // nb column slots: X_ij, i >= j
  if (a.out[1] != 1.0) return;
  double* sAl = sXcol + (size_t)a.nb * 256;        // kTriWaves x 16: alpha's parts
  const int nb = a.nb, j = blockIdx.x, lane = threadIdx.x & 63, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  TriState<R> st;
  // u_i[4s + g] of the wave's rows and of row j (wave 0), loaded up front
  // unless the registers are wanted for the ring
  double uv[R + 1][4];
  auto load_u = [&]() {
#pragma unroll
    for (int t = 0; t <= R; ++t) {
      const int i = t < R ? j + 1 + wave + kTriWaves * t : j;
#pragma unroll
      for (int s = 0; s < 4; ++s) uv[t][s] = i < nb ? a.u[16 * i + 4 * s + g] : 0.0;
    }
  };
  if constexpr (R <= 4) load_u();
#pragma unroll
  for (int t = 0; t < R; ++t) {
    st.S[t] = zero4();
    const int i = j + 1 + wave + kTriWaves * t;
#pragma unroll
    for (int b = 0; b < kTriAhead; ++b)
      ld_cols(a.L + (i < nb && j + b < i ? ((size_t)i * nb + j + b) * 256 : 0), lane, st.Lv[b][t]);
    ld_rows(a.Di + (i < nb ? (size_t)i * 256 : 0), lane, st.Dv[t]);
  }
  if (wave == 0) st_col_slot(sXcol + (size_t)j * 256, ld_c(a.Di + (size_t)j * 256, lane), lane);
  // all of the above in registers before the loop, so that inside it a wait
  // is only ever for the ring slot about to be used
  __builtin_amdgcn_s_waitcnt(0);
  lds_barrier();
  for (int k = j; k + 1 < nb; k += kTriAhead) {
    tri_step<R, 0>(a, st, sXcol, j, k, wave, lane);
    tri_step<R, 1>(a, st, sXcol, j, k + 1, wave, lane);
    tri_step<R, 2>(a, st, sXcol, j, k + 2, wave, lane);
  }
  // the column, row-major blocks
  for (int i = j + wave; i < nb; i += kTriWaves) {
    double x[4];
    ld_slot(sXcol + (size_t)i * 256, lane, x);
    st_c(a.Xi + ((size_t)i * nb + j) * 256, d4_t{x[0], x[1], x[2], x[3]}, lane);
  }
  // alpha_j = sum_{i >= j} X_ij^T u_i (alpha = L^-T L^-1 r): each wave its rows,
  // then the waves in order
  if constexpr (R > 4) load_u();
  double acc = 0.0;
#pragma unroll
  for (int t = 0; t <= R; ++t) {
    const int i = t < R ? j + 1 + wave + kTriWaves * t : j;
    if (i < nb && (t < R || wave == 0)) {
      double x[4];
      ld_slot(sXcol + (size_t)i * 256, lane, x);  // X_ij[4s + g][c]
#pragma unroll
      for (int s = 0; s < 4; ++s) acc = fma(x[s], uv[t][s], acc);
    }
  }
  acc += __shfl_xor(acc, 16);
  acc += __shfl_xor(acc, 32);
  if (lane < 16) sAl[wave * 16 + lane] = acc;
  lds_barrier();
  if (wave == 0 && lane < 16) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < kTriWaves; ++w) s += sAl[w * 16 + lane];
    a.alpha[16 * j + lane] = s;
  }
}

// ---- kernel B: the gradient's partial sums, one lower block per workgroup ---
// Z_IJ = (K^-1)_IJ = sum_{k >= I} X_kI^T X_kJ on the matrix cores (wave w
// takes k = I + w, I + w + 4, ...; the four sums are added in order through
// LDS, and a diagonal block is made exactly symmetric), then one element of
// W = alpha alpha^T - K^-1 per thread with the covariance and its
// derivatives recomputed.
template <int D, bool LW>
__global__ __launch_bounds__(kGradThreads) void nll_grad_kernel(NllArgs a) {
  constexpr int P = LW ? 3 * D + 2 : D + 2;
  __shared__ double sZ[kGradWaves][256];
  __shared__ double sRed[kGradWaves][P];
  if (a.out[1] != 1.0) return;  // K not positive definite: no gradient
  const int nb = a.nb, m = a.m, t = threadIdx.x, lane = t & 63, wave = t >> 6;
  int I = 0, J = 0;
  advance_lower(I, J, blockIdx.x);
  d4_t Zv = zero4();
  for (int k0 = I + wave; k0 < nb; k0 += 4 * kGradWaves) {
    double av[4][4], bv[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int k = k0 + u * kGradWaves;
      if (k < nb) {
        ld_cols(a.Xi + ((size_t)k * nb + I) * 256, lane, av[u]);  // X_kI^T as an A operand
        ld_cols(a.Xi + ((size_t)k * nb + J) * 256, lane, bv[u]);  // X_kJ as a B operand
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (k0 + u * kGradWaves < nb) Zv = mma16(Zv, av[u], bv[u]);
  }
  st_c(sZ[wave], Zv, lane);
  __syncthreads();
  const int ii = t >> 4, jj = t & 15, i = 16 * I + ii, j = 16 * J + jj;
  double zij = ((sZ[0][t] + sZ[1][t]) + sZ[2][t]) + sZ[3][t];
  if (I == J) {
    const int tt = jj * 16 + ii;
    zij = 0.5 * (zij + (((sZ[0][tt] + sZ[1][tt]) + sZ[2][tt]) + sZ[3][tt]));
  }
  double g[P];
#pragma unroll
  for (int p = 0; p < P; ++p) g[p] = 0.0;
  if (!((I == J && jj > ii) || i >= m || j >= m)) {
    const bool m52 = a.m52 != 0;
    const double s2 = exp(a.theta[D]), tau2 = exp(a.theta[D + 1]);
    const double root = m52 ? kRoot5 : kRoot3;
    const double* X = LW ? a.Xw : a.X;
    const double w = 0.5 * (i == j ? 1.0 : 2.0) * (a.alpha[i] * a.alpha[j] - zij);  // W and dK are symmetric
    double tk[D], inv_ls[D], r2 = 0.0;
#pragma unroll
    for (int k = 0; k < D; ++k) {
      inv_ls[k] = exp(-a.theta[k]);
      tk[k] = (X[(size_t)i * D + k] - X[(size_t)j * D + k]) * inv_ls[k];
      r2 += tk[k] * tk[k];
    }
    const double tt = root * sqrt(r2), e = exp(-tt);
    const double kv = matern(m52, s2, tt, e);
    const double rad = m52 ? 5.0 / 3.0 * s2 * (1.0 + tt) * e : 3.0 * s2 * e;
    const double wr = w * rad;
#pragma unroll
    for (int k = 0; k < D; ++k) {
      g[k] -= wr * (tk[k] * tk[k]);
      if constexpr (LW) {
        const double wt = wr * tk[k] * inv_ls[k];
        g[D + 2 + k] += wt * (a.Ga[(size_t)i * D + k] - a.Ga[(size_t)j * D + k]);
        g[2 * D + 2 + k] += wt * (a.Gb[(size_t)i * D + k] - a.Gb[(size_t)j * D + k]);
      }
    }
    g[D] -= w * kv;
    if (i == j) g[D + 1] -= w * tau2;
  }
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const double v = wave_sum(g[p]);
    if (lane == 0) sRed[wave][p] = v;
  }
  __syncthreads();
  if (t < P) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < kGradWaves; ++w) s += sRed[w][t];
    a.hout[1 + 17 * nb + (size_t)blockIdx.x * P + t] = s;
  }
}

template <int D, typename F>
int by_dim(int d, F&& f) {
  if constexpr (D > SCOOT_MAX_DIM) {
    return fail(SCOOT_ERR_UNSUPPORTED, "gp nll: d exceeds SCOOT_MAX_DIM");
  } else {
    if (d == D) return f(std::integral_constant<int, D>());
    return by_dim<D + 1>(d, std::forward<F>(f));
  }
}

// Device state of one likelihood (one objective): inputs, work matrices and a
// pinned read-back buffer, all allocated once per search.
class DeviceNll {
 public:
  ~DeviceNll() {
    if (buf_) (void)hipFree(buf_);
    if (host_) (void)hipHostFree(host_);
  }
  int init(const std::vector<double>& X, const std::vector<double>& r, int m, int d, scoot_kernel kernel,
           bool learn_warp, hipStream_t s) {
    s_ = s;
    m_ = m;
    d_ = d;
    lw_ = learn_warp;
    P_ = learn_warp ? 3 * d + 2 : d + 2;
    nb_ = (m + 15) / 16;
    // every part 256-byte aligned (32 doubles)
    auto up = [](size_t n) { return (n + 31) / 32 * 32; };
    const size_t md = (size_t)m * d, mp = (size_t)nb_ * 16, blocks = (size_t)nb_ * nb_ * 256;
    const size_t n = up(md) + up(mp) + 2 * blocks + (size_t)nb_ * 256 + (learn_warp ? 3 * up(md) : 0) +
                     2 * up(mp) + up(2);
    if (hipMalloc(&buf_, n * sizeof(double)) != hipSuccess) {
      buf_ = nullptr;
      return fail(SCOOT_ERR_NO_MEMORY, "gp nll: device allocation failed");
    }
    // the results, written by the kernels straight into coherent pinned host
    // memory (no copy after them): status, pivot products, u, partial gradient
    // sums
    n_lower_ = nb_ * (nb_ + 1) / 2;
    if (hipHostMalloc(&host_, (1 + 17 * (size_t)nb_ + (size_t)n_lower_ * P_) * sizeof(double),
                      hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess) {
      host_ = nullptr;
      return fail(SCOOT_ERR_NO_MEMORY, "gp nll: pinned allocation failed");
    }
    void* hdev = nullptr;
    if (hipHostGetDevicePointer(&hdev, host_, 0) != hipSuccess || hdev == nullptr)
      return fail(SCOOT_ERR_DEVICE, "gp nll: pinned memory not visible to the device");
    a_.hout = static_cast<double*>(hdev);
    double* p = buf_;
    double* Xd = p;
    p += up(md);
    double* rd = p;
    p += up(mp);
    a_.L = p;
    p += blocks;
    a_.Xi = p;
    p += blocks;
    a_.Di = p;
    p += (size_t)nb_ * 256;
    a_.Xw = a_.Ga = a_.Gb = nullptr;
    if (learn_warp) {
      a_.Xw = p;
      a_.Ga = p + up(md);
      a_.Gb = p + 2 * up(md);
      p += 3 * up(md);
    }
    a_.alpha = p;
    p += up(mp);
    a_.u = p;
    p += up(mp);
    a_.out = p;
    a_.X = Xd;
    a_.r = rd;
    a_.m = m;
    a_.nb = nb_;
    a_.d = d;
    a_.m52 = kernel == SCOOT_MATERN52;
    a_.learn_warp = learn_warp;
    std::vector<double> rp(mp, 0.0);
    std::memcpy(rp.data(), r.data(), sizeof(double) * m);
    if (hipMemcpyAsync(Xd, X.data(), md * sizeof(double), hipMemcpyHostToDevice, s) != hipSuccess ||
        hipMemcpyAsync(rd, rp.data(), mp * sizeof(double), hipMemcpyHostToDevice, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      return fail(SCOOT_ERR_DEVICE, std::string("gp nll: upload failed: ") + hipGetErrorString(hipGetLastError()));
    lds_ = ((size_t)nb_ * 512 + 256 + 512 + SCOOT_MAX_OBS / 16 + (size_t)nb_ * 16 + 32) * sizeof(double) +
           (4 + kNllWaves + (size_t)nb_ * (nb_ - 1) / 2) * sizeof(int);

    int rc = allow_full_lds((const void*)nll_factor_kernel, "gp nll");
    const void* tri[] = {(const void*)nll_trtri_kernel<1>, (const void*)nll_trtri_kernel<2>,
                         (const void*)nll_trtri_kernel<3>, (const void*)nll_trtri_kernel<4>,
                         (const void*)nll_trtri_kernel<kTriMaxRows>};
    for (const void* f : tri)
      if (rc == SCOOT_OK) rc = allow_full_lds(f, "gp nll");
    return rc;
  }
  // false when K is not positive definite; a device failure is kept in error().
  bool eval(const double* theta, double* nll, double* grad) {
    if (rc_ != SCOOT_OK) return false;
    std::memcpy(a_.theta, theta, sizeof(double) * P_);
    (void)hipGetLastError();  // clear an earlier, unrelated error
    if (lw_)
      hipLaunchKernelGGL(nll_warp_kernel, dim3((unsigned)((m_ * d_ + 255) / 256)), dim3(256), 0, s_, a_);
    hipLaunchKernelGGL(nll_cov_kernel, dim3((unsigned)(nb_ * (nb_ + 1) / 2)), dim3(256), 0, s_, a_);
    hipLaunchKernelGGL(nll_factor_kernel, dim3(1), dim3(kNllThreads), lds_, s_, a_);
    if (grad) {  // L^-1 and alpha, then K^-1 and the gradient's partial sums (the NLL needs none of them)
      launch_trtri();
      const int rc = by_dim<1>(d_, [&](auto D) {
        if (lw_)
          hipLaunchKernelGGL((nll_grad_kernel<decltype(D)::value, true>), dim3((unsigned)n_lower_), dim3(kGradThreads), 0,
                             s_, a_);
        else
          hipLaunchKernelGGL((nll_grad_kernel<decltype(D)::value, false>), dim3((unsigned)n_lower_), dim3(kGradThreads), 0,
                             s_, a_);
        return SCOOT_OK;
      });
      if (rc != SCOOT_OK) {
        rc_ = rc;
        return false;
      }
    }
    const hipError_t launched = hipGetLastError();
    if (launched != hipSuccess) {
      rc_ = fail(SCOOT_ERR_DEVICE, std::string("gp nll: launch failed: ") + hipGetErrorString(launched));
      return false;
    }
    if (hipStreamSynchronize(s_) != hipSuccess) {
      rc_ = fail(SCOOT_ERR_DEVICE, std::string("gp nll: device evaluation failed: ") +
                                       hipGetErrorString(hipGetLastError()));
      return false;
    }
    if (host_[0] == 2.0) {
      rc_ = fail(SCOOT_ERR_DEVICE, "gp nll: the factorization's wait for its diagonal block ran out");
      return false;
    }
    if (host_[0] != 1.0) return false;
    // NLL = 1/2 |L^-1 r|^2 + 1/2 log det K + m/2 log(2 pi), and the gradient's
    // partial sums, each added in a fixed order
    double q = 0.0, logdet = 0.0;
    for (int k = 0; k < nb_; ++k) logdet += std::log(host_[1 + k]);
    for (int i = 0; i < 16 * nb_; ++i) q += host_[1 + nb_ + i] * host_[1 + nb_ + i];
    *nll = 0.5 * q + 0.5 * logdet + 0.5 * m_ * kLog2PiD;
    if (grad) {
      const double* part = host_ + 1 + 17 * nb_;
      for (int p = 0; p < P_; ++p) {
        double s = 0.0;
        for (int b = 0; b < n_lower_; ++b) s += part[(size_t)b * P_ + p];
        grad[p] = s;
      }
    }
    return true;
  }
  // K, the factor and L^-1 at theta, then L^-1 (m x m row-major, lower) and
  // alpha to the host; false when K is not positive definite or on a device
  // failure (kept in error()).
  bool inverse(const double* theta, std::vector<double>& Linv, std::vector<double>& alpha) {
    if (rc_ != SCOOT_OK) return false;
    std::memcpy(a_.theta, theta, sizeof(double) * P_);
    (void)hipGetLastError();  // clear an earlier, unrelated error
    if (lw_)
      hipLaunchKernelGGL(nll_warp_kernel, dim3((unsigned)((m_ * d_ + 255) / 256)), dim3(256), 0, s_, a_);
    hipLaunchKernelGGL(nll_cov_kernel, dim3((unsigned)(nb_ * (nb_ + 1) / 2)), dim3(256), 0, s_, a_);
    hipLaunchKernelGGL(nll_factor_kernel, dim3(1), dim3(kNllThreads), lds_, s_, a_);
    launch_trtri();
    const hipError_t launched = hipGetLastError();
    if (launched != hipSuccess) {
      rc_ = fail(SCOOT_ERR_DEVICE, std::string("gp fit: launch failed: ") + hipGetErrorString(launched));
      return false;
    }
    if (hipStreamSynchronize(s_) != hipSuccess) {
      rc_ = fail(SCOOT_ERR_DEVICE, std::string("gp fit: device factorization failed: ") +
                                       hipGetErrorString(hipGetLastError()));
      return false;
    }
    if (host_[0] == 2.0) {
      rc_ = fail(SCOOT_ERR_DEVICE, "gp fit: the factorization's wait for its diagonal block ran out");
      return false;
    }
    if (host_[0] != 1.0) return false;
    std::vector<double> xi((size_t)nb_ * nb_ * 256), al((size_t)nb_ * 16);
    if (hipMemcpyAsync(xi.data(), a_.Xi, xi.size() * sizeof(double), hipMemcpyDeviceToHost, s_) != hipSuccess ||
        hipMemcpyAsync(al.data(), a_.alpha, al.size() * sizeof(double), hipMemcpyDeviceToHost, s_) != hipSuccess ||
        hipStreamSynchronize(s_) != hipSuccess) {
      rc_ = fail(SCOOT_ERR_DEVICE, std::string("gp fit: read-back failed: ") + hipGetErrorString(hipGetLastError()));
      return false;
    }
    const int m = m_;
    Linv.assign((size_t)m * m, 0.0);
    for (int row = 0; row < m; ++row)
      for (int col = 0; col <= row; ++col) {
        const int I = row >> 4, J = col >> 4;
        Linv[(size_t)row * m + col] = xi[((size_t)I * nb_ + J) * 256 + (row & 15) * 16 + (col & 15)];
      }
    alpha.assign(al.begin(), al.begin() + m);
    return true;
  }
  int error() const { return rc_; }

 private:
  void launch_trtri() {
    const size_t lds_tri = ((size_t)nb_ * 256 + kTriWaves * 16) * sizeof(double);
    switch ((nb_ - 1 + kTriWaves - 1) / kTriWaves) {
      case 0:
      case 1: hipLaunchKernelGGL(nll_trtri_kernel<1>, dim3((unsigned)nb_), dim3(kTriWaves * 64), lds_tri, s_, a_); break;
      case 2: hipLaunchKernelGGL(nll_trtri_kernel<2>, dim3((unsigned)nb_), dim3(kTriWaves * 64), lds_tri, s_, a_); break;
      case 3: hipLaunchKernelGGL(nll_trtri_kernel<3>, dim3((unsigned)nb_), dim3(kTriWaves * 64), lds_tri, s_, a_); break;
      case 4: hipLaunchKernelGGL(nll_trtri_kernel<4>, dim3((unsigned)nb_), dim3(kTriWaves * 64), lds_tri, s_, a_); break;
      default: hipLaunchKernelGGL(nll_trtri_kernel<kTriMaxRows>, dim3((unsigned)nb_), dim3(kTriWaves * 64), lds_tri, s_, a_);
    }
  }
  hipStream_t s_ = nullptr;
  int m_ = 0, d_ = 0, nb_ = 0, n_lower_ = 0, P_ = 0;
  bool lw_ = false;
  size_t lds_ = 0;
  double* buf_ = nullptr;
  double* host_ = nullptr;
  NllArgs a_{};
  int rc_ = SCOOT_OK;
};

int device_inputs(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                  const double* warp_b, double c, bool learn_warp, std::vector<double>& Xu, std::vector<double>& r) {
  if (learn_warp && (warp_a || warp_b))
    return fail(SCOOT_ERR_INVALID_ARG, "gp nll: a learned warp takes no fixed warp_a / warp_b");
  return mle_inputs(X, y, m, d, kernel, warp_a, warp_b, c, learn_warp, Xu, r);
}

}  // namespace

int mle_nll_device(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                   const double* warp_b, double c, bool learn_warp, const double* theta, double* nll, double* grad,
                   void* stream) {
  if (!theta || !nll) return fail(SCOOT_ERR_INVALID_ARG, "gp nll: null pointer");
  std::vector<double> Xu, r;
  int rc = device_inputs(X, y, m, d, kernel, warp_a, warp_b, c, learn_warp, Xu, r);
  if (rc != SCOOT_OK) return rc;
  const int P = learn_warp ? 3 * d + 2 : d + 2;
  for (int k = 0; k < P; ++k)
    if (!std::isfinite(theta[k])) return fail(SCOOT_ERR_INVALID_ARG, "gp nll: non-finite theta");
  DeviceNll dev;
  rc = dev.init(Xu, r, m, d, kernel, learn_warp, (hipStream_t)stream);
  if (rc != SCOOT_OK) return rc;
  const bool ok = dev.eval(theta, nll, grad);
  if (dev.error() != SCOOT_OK) return dev.error();
  if (!ok) return fail(SCOOT_ERR_NOT_PD, "gp nll: K is not positive definite");
  return SCOOT_OK;
}

int mle_fit_device(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                   const double* warp_b, double c, bool learn_warp, const double* lower, const double* upper,
                   int max_iter, double* theta, double* nll_out, int* iters_out, void* stream) {
  std::vector<double> Xu, r;
  int rc = device_inputs(X, y, m, d, kernel, warp_a, warp_b, c, learn_warp, Xu, r);
  if (rc != SCOOT_OK) return rc;
  DeviceNll dev;
  rc = dev.init(Xu, r, m, d, kernel, learn_warp, (hipStream_t)stream);
  if (rc != SCOOT_OK) return rc;
  rc = lbfgs_box([&](const double* t, double* f, double* g) { return dev.eval(t, f, g); },
                 learn_warp ? 3 * d + 2 : d + 2, lower, upper, max_iter, theta, nll_out, iters_out);
  if (dev.error() != SCOOT_OK) return dev.error();
  return rc;
}

namespace {
// The GP at theta from a factorization on dev: the host part of a fit, then
// L^-1 and alpha from the device.
int gp_from_device(DeviceNll& dev, const double* X, const double* y, int m, int d, scoot_kernel kernel,
                   const double* warp_a, const double* warp_b, double c, bool learn_warp, const double* theta,
                   scoot_dtype dt, scoot_gp* out) {
  double ls[SCOOT_MAX_DIM], wa[SCOOT_MAX_DIM], wb[SCOOT_MAX_DIM];
  for (int k = 0; k < d; ++k) ls[k] = std::exp(theta[k]);
  const double* pa = warp_a;
  const double* pb = warp_b;
  if (learn_warp) {
    for (int k = 0; k < d; ++k) {
      wa[k] = std::exp(theta[d + 2 + k]);
      wb[k] = std::exp(theta[2 * d + 2 + k]);
    }
    pa = wa;
    pb = wb;
  }
  FitHost f;
  int rc = fit_setup(X, y, m, d, kernel, ls, pa, pb, std::exp(theta[d]), std::exp(theta[d + 1]), c, f);
  if (rc != SCOOT_OK) return rc;
  if (!dev.inverse(theta, f.Linv, f.alpha))
    return dev.error() != SCOOT_OK ? dev.error()
                                   : fail(SCOOT_ERR_NOT_PD, "gp fit: K + tau^2 I is not positive definite");
  return gp_from_fit(f, pa, pb, dt, out);
}
}  // namespace

int mle_fit_device_gp(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                      const double* warp_b, double c, bool learn_warp, const double* lower, const double* upper,
                      int max_iter, double* theta, scoot_dtype dt, void* stream, scoot_gp* out) {
  std::vector<double> Xu, r;
  int rc = device_inputs(X, y, m, d, kernel, warp_a, warp_b, c, learn_warp, Xu, r);
  if (rc != SCOOT_OK) return rc;
  DeviceNll dev;
  rc = dev.init(Xu, r, m, d, kernel, learn_warp, (hipStream_t)stream);
  if (rc != SCOOT_OK) return rc;
  rc = lbfgs_box([&](const double* t, double* f, double* g) { return dev.eval(t, f, g); },
                 learn_warp ? 3 * d + 2 : d + 2, lower, upper, max_iter, theta, nullptr, nullptr);
  if (dev.error() != SCOOT_OK) return dev.error();
  if (rc != SCOOT_OK) return rc;
  return gp_from_device(dev, X, y, m, d, kernel, warp_a, warp_b, c, learn_warp, theta, dt, out);
}

int gp_fit_device(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* ls,
                  const double* warp_a, const double* warp_b, double s2, double tau2, double c, scoot_dtype dt,
                  void* stream, scoot_gp* out) {
  if (!ls) return fail(SCOOT_ERR_INVALID_ARG, "gp fit: null pointer");
  if (d < 1 || d > SCOOT_MAX_DIM) return fail(SCOOT_ERR_INVALID_ARG, "gp fit: bad d");
  for (int k = 0; k < d; ++k)
    if (!(ls[k] > 0) || !std::isfinite(ls[k]))
      return fail(SCOOT_ERR_INVALID_ARG, "gp fit: lengthscales must be finite and > 0");
  if (!(s2 > 0) || !std::isfinite(s2) || !(tau2 > 0) || !std::isfinite(tau2))
    return fail(SCOOT_ERR_INVALID_ARG, "gp fit (device): signal and noise variance must be finite and > 0");
  double theta[SCOOT_MAX_DIM + 2];
  for (int k = 0; k < d; ++k) theta[k] = std::log(ls[k]);
  theta[d] = std::log(s2);
  theta[d + 1] = std::log(tau2);
  std::vector<double> Xu, r;
  int rc = device_inputs(X, y, m, d, kernel, warp_a, warp_b, c, false, Xu, r);
  if (rc != SCOOT_OK) return rc;
  DeviceNll dev;
  rc = dev.init(Xu, r, m, d, kernel, false, (hipStream_t)stream);
  if (rc != SCOOT_OK) return rc;
  return gp_from_device(dev, X, y, m, d, kernel, warp_a, warp_b, c, false, theta, dt, out);
}

}  // namespace scoot
