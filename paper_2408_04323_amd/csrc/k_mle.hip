// The GP's negative log likelihood and its gradient in the hyperparameters,
// evaluated on the device in fp64 (Sec. 4.3: the noise level and the other
// hyperparameters are learned by maximum likelihood).  The search itself (the
// box-constrained L-BFGS of host_mle.cpp) stays on the host and calls this
// once per trial point.
//
// With r = y - c, K = k_theta(X, X) + tau2 I (m x m) and W = alpha alpha^T - K^-1:
//   NLL = 1/2 r^T alpha + 1/2 log det K + m/2 log(2 pi),   alpha = K^-1 r
//   dNLL/dtheta_p = -1/2 sum_ij W_ij (dK/dtheta_p)_ij
// with the derivatives of the covariance written out in host_mle.cpp.
//
// Matrices are 16 x 16 blocks (row-major inside a block), m padded to a
// multiple of 16 with identity rows (their covariance with real rows is 0,
// their diagonal 1, their r 0: log det, the quadratic form and the gradient do
// not see them).  The kernels of one evaluation, on one stream:
//   W. (warp learned) the warped inputs and their derivatives;
//   K. K, one 16 x 16 block per workgroup;
//   A. one workgroup (8 waves): the Cholesky factor L by 16-column block
//      steps: the diagonal block by one wave in registers, the panel below it
//      by forward substitution (a row per thread), the trailing update on
//      v_mfma_f64_16x16x4f64; the next diagonal block is factored as soon as
//      it is updated, by a wave whose SIMD the others leave free; then the
//      inverses of the diagonal blocks;
//   T. L^-1, one block column per workgroup (the columns are independent);
//   U. K^-1 = L^-T L^-1, one block per workgroup;
//   V. alpha = K^-1 r and the quadratic form, one block row per workgroup;
//   B. the gradient: one element of W per thread, the covariance and its
//      derivatives recomputed, partial sums per workgroup;
//   C. the NLL and the gradient's partial sums, added in a fixed order.
// Every operation is in double and every sum has a fixed order, so an
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
constexpr int kGradBlocks = 64;
constexpr int kGradThreads = 256;
constexpr double kRoot5 = 2.23606797749978969641;
constexpr double kRoot3 = 1.73205080756887729353;
constexpr double kLog2PiD = 1.83787706640934548356;

struct NllArgs {
  const double* X;  // m x d inputs as the covariance sees them (raw when the warp is learned)
  const double* r;  // m_pad: y - c, 0 beyond m
  double* L;        // nb x nb blocks: K, then its lower factor (blocks I >= J)
  double* Z;        // nb x nb blocks: K^-1 (blocks I >= J)
  double* Xi;       // nb x nb blocks: L^-1 (blocks I >= J)
  double* Di;       // nb blocks: inverses of L's diagonal blocks
  double* Xw;       // m x d warped inputs (warp learned)
  double* Ga;       // m x d: d w / d log a (warp learned)
  double* Gb;       // m x d: d w / d log b (warp learned)
  double* alpha;    // m_pad
  double* prod;     // nb: product of each diagonal block's pivots (real rows)
  double* qpart;    // nb: r^T alpha over each block of 16 rows
  double* out;      // [0] NLL, [1] 1 when K is numerically positive definite else 0, [2 ..] gradient
  double* part;     // kGradBlocks x P partial gradient sums
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
  const int ii = t >> 4, jj = t & 15, i = 16 * I + ii, j = 16 * J + jj;
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

// Factors the 16 x 16 diagonal block kk in one wave: stores L_kk (row-major,
// zero above the diagonal) to memory and to sL (16 x 17), 1 / L[c][c] to
// sIc, the product of the pivots of real rows to sProd[kk]; raises sFlag when
// such a pivot is not above floor (or a padding pivot is not positive).
//
// In: lane l holds column jl = l % 16 of the block, col[i] = A[i][jl] (each row
// of 16 lanes a copy).  Step c takes the pivot from lane c; by the block's
// symmetry lane j finds its entry of column c, L[j][c] = A[c][j] / L[c][c], in
// its own registers, and the column goes to every lane entry by entry
// (readlane) for the update of the columns right of c (lanes j <= c are
// finished and their registers no longer read).
__device__ inline void diag_step(const NllArgs& a, int kk, double (&col)[16], double* sL, double* sIc,
                                 double* sProd, int* sFlag, double floor, int lane) {
  const int jl = lane & 15, real = min(16, a.m - 16 * kk);
  double row[16], prod = 1.0;
  bool bad = false;
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    const double piv = lane_bcast(col[c], c);
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
    const double lj = col[c] * ic;
    row[c] = jl == c ? piv * ic : lj;
    if (lane == c) sIc[c] = ic;
#pragma unroll
    for (int i = c + 1; i < 16; ++i) {
      col[i] = fma(-lane_bcast(lj, i), lj, col[i]);
      __builtin_amdgcn_sched_barrier(0);  // each broadcast used where it is made
    }
  }
  if (lane < 16) {
    double* Lb = a.L + ((size_t)kk * a.nb + kk) * 256 + jl * 16;
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const double v = c <= jl ? row[c] : 0.0;
      Lb[c] = v;
      sL[jl * 17 + c] = v;
    }
  }
  if (lane == 0) {
    sProd[kk] = prod;
    if (bad) sFlag[0] = 1;
  }
}

// ---- kernel A: L, K^-1, alpha, NLL --------------------------------------------
__global__ __launch_bounds__(kNllThreads) void nll_factor_kernel(NllArgs a) {
  extern __shared__ __align__(16) double sm[];
  const int nb = a.nb, m = a.m, d = a.d;
  double* sPan = sm;                          // nb slots: the panel (row slots), a column of L (column slots)
  double* sLkk = sPan + (size_t)nb * 256;     // 16 x 17: the current diagonal block's factor
  double* sIc = sLkk + 16 * 17;               // 16: 1 / its pivots' roots
  double* sScr = sIc + 16;                    // 256: wave 0's scratch, a block read by columns
  double* sProd = sScr + 256;                 // per diagonal block: product of its pivots
  double* sRed = sProd + SCOOT_MAX_OBS / 16;  // kNllWaves
  int* sFlag = reinterpret_cast<int*>(sRed + kNllWaves);
  int* sSimd = sFlag + 4;                     // kNllWaves: the SIMD each wave runs on

  const int tid = threadIdx.x, lane = tid & 63, jl = lane & 15;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if (lane == 0) sSimd[wave] = (int)((__builtin_amdgcn_s_getreg((31 << 11) | 4) >> 4) & 3);  // HW_ID.SIMD_ID
  const double s2 = exp(a.theta[d]), tau2 = exp(a.theta[d + 1]);
  // A pivot that is not above 1e-13 of its original diagonal entry (s2 + tau2)
  // means K is not numerically positive definite (the host factor's rule).
  const double floor = 1e-13 * (s2 + tau2);

  // ---- Cholesky factor, 16 columns per step --------------------------------
  // Step k: the panel L_ik = A_ik L_kk^-T (matrix cores), then the trailing
  // update A_ij -= L_ik L_jk^T; the wave that updates block (k+1, k+1) factors
  // it at once, while the others update the rest.
  if (wave == 0) {
    if (lane == 0) sFlag[0] = 0;
    double col[16];
    const double* blk = a.L;
#pragma unroll
    for (int i = 0; i < 16; ++i) col[i] = blk[i * 16 + jl];
    diag_step(a, 0, col, sLkk, sIc, sProd, sFlag, floor, lane);
  }
  __syncthreads();
  // The trailing update goes to the waves that do not share wave 0's SIMD:
  // the vector ALU wave 0 factors with and the matrix unit are one datapath,
  // so a neighbour's matrix instructions would stall the factorization.
  int worker = -1, n_workers = 0;
  for (int w = 1; w < kNllWaves; ++w)
    if (sSimd[w] != sSimd[0]) {
      if (w == wave) worker = n_workers;
      ++n_workers;
    }
  bool failed = false;
  for (int k = 0; k < nb; ++k) {
    if (sFlag[0]) {
      failed = true;
      break;
    }
    // panel: L_ik = A_ik L_kk^-T, one row per thread (forward substitution)
    const int rows = (nb - k - 1) * 16;
    for (int ri = tid; ri < rows; ri += kNllThreads) {
      const int ib = k + 1 + (ri >> 4), rr = ri & 15;
      double* rowp = a.L + ((size_t)ib * nb + k) * 256 + rr * 16;
      double x[16];
#pragma unroll
      for (int c = 0; c < 16; c += 2) {
        const d2_t v = *reinterpret_cast<const d2_t*>(rowp + c);
        x[c] = v[0], x[c + 1] = v[1];
      }
#pragma unroll
      for (int c = 0; c < 16; ++c) {
        x[c] *= sIc[c];
#pragma unroll
        for (int q = c + 1; q < 16; ++q) x[q] = fma(-x[c], sLkk[q * 17 + c], x[q]);
      }
      double* slot = sPan + (size_t)ib * 256;
#pragma unroll
      for (int c = 0; c < 16; c += 2) *reinterpret_cast<d2_t*>(rowp + c) = d2_t{x[c], x[c + 1]};
#pragma unroll
      for (int c = 0; c < 16; ++c) slot[row_slot_pos(rr, c)] = x[c];
    }
    __syncthreads();
    if (k == nb - 1) break;
    if (wave == 0) {
      const int i = k + 1;
      double* blk = a.L + ((size_t)i * nb + i) * 256;
      d4_t acc = ld_c(blk, lane);
      double av[4], bv[4];
      ld_slot(sPan + (size_t)i * 256, lane, bv);
#pragma unroll
      for (int s = 0; s < 4; ++s) av[s] = -bv[s];
      acc = mma16(acc, av, bv);
      st_c(sScr, acc, lane);  // row-major, to read by columns
      wave_lds_sync();
      double col[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) col[r] = sScr[r * 16 + jl];
      diag_step(a, i, col, sLkk, sIc, sProd, sFlag, floor, lane);
    } else if (worker >= 0) {
      // blocks 1, 2, ... of the trailing triangle (row by row) over the
      // workers, four per wave at a time, their loads issued first
      const int W = n_workers;
      const int T = nb - k - 1, n_trail = T * (T + 1) / 2;
      int I = 0, J = 0;
      advance_lower(I, J, 1 + worker);
      for (int b = 1 + worker; b < n_trail; b += 4 * W) {
        d4_t acc[4];
        double* blk[4];
        int bi[4], bj[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          bi[u] = k + 1 + I;
          bj[u] = k + 1 + J;
          blk[u] = a.L + ((size_t)bi[u] * nb + bj[u]) * 256;
          if (b + u * W < n_trail) acc[u] = ld_c(blk[u], lane);
          advance_lower(I, J, W);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (b + u * W < n_trail) {
            double av[4], bv[4];
            ld_slot(sPan + (size_t)bi[u] * 256, lane, av);
            ld_slot(sPan + (size_t)bj[u] * 256, lane, bv);
#pragma unroll
            for (int s = 0; s < 4; ++s) av[s] = -av[s];
            st_c(blk[u], mma16(acc[u], av, bv), lane);
          }
        }
      }
    }
    __syncthreads();
  }

  if (tid == 0) a.out[1] = failed ? 0.0 : 1.0;
  if (failed) return;
  if (tid < nb) a.prod[tid] = sProd[tid];
  // inverses of the diagonal blocks, one column per lane of a group of 16
  const int grp = tid >> 4, q = tid & 15;
  for (int jb = grp; jb < nb; jb += kNllThreads / 16) {
    const double* Lb = a.L + ((size_t)jb * nb + jb) * 256;
    double x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      double acc = i == q ? 1.0 : 0.0;
#pragma unroll
      for (int t = 0; t < i; ++t) acc = fma(-Lb[i * 16 + t], x[t], acc);
      x[i] = acc / Lb[i * 16 + i];
    }
    double* Db = a.Di + (size_t)jb * 256;
#pragma unroll
    for (int i = 0; i < 16; ++i) Db[i * 16 + q] = x[i];
  }
}

// ---- kernel T: L^-1, one block column per workgroup ---------------------------
// Column j: X_jj = Di_j, then for i = j+1 .. nb-1
//   X_ij = -Di_i sum_{k=j}^{i-1} L_ik X_kj,
// the sum split over the four waves (added in wave order), X's column kept in
// LDS as column slots for the next rows.
constexpr int kTriWaves = 4;
__global__ __launch_bounds__(kTriWaves * 64) void nll_trtri_kernel(NllArgs a) {
  extern __shared__ __align__(16) double sm[];
  if (a.out[1] != 1.0) return;
  const int nb = a.nb, j = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  double* sX = sm;                            // nb column slots: X_kj
  double* sPart = sX + (size_t)nb * 256;      // kTriWaves column slots: partial sums
  if (wave == 0) {
    const d4_t v = ld_c(a.Di + (size_t)j * 256, lane);
    st_col_slot(sX + (size_t)j * 256, v, lane);
    st_c(a.Xi + ((size_t)j * nb + j) * 256, v, lane);
  }
  __syncthreads();
  for (int i = j + 1; i < nb; ++i) {
    d4_t S = zero4();
    for (int k = j + wave; k < i; k += kTriWaves) {
      double av[4], bv[4];
      ld_rows(a.L + ((size_t)i * nb + k) * 256, lane, av);
      ld_slot(sX + (size_t)k * 256, lane, bv);
      S = mma16(S, av, bv);
    }
    st_col_slot(sPart + wave * 256, S, lane);
    __syncthreads();
    if (wave == 0) {
      d4_t T = zero4();
      for (int w = 0; w < kTriWaves; ++w) {
        double pv[4];
        ld_slot(sPart + w * 256, lane, pv);
#pragma unroll
        for (int r = 0; r < 4; ++r) T[r] += pv[r];
      }
      double av[4];
      ld_rows(a.Di + (size_t)i * 256, lane, av);
#pragma unroll
      for (int s = 0; s < 4; ++s) av[s] = -av[s];
      const double tb[4] = {T[0], T[1], T[2], T[3]};  // T as a B operand is its own C layout
      const d4_t v = mma16(zero4(), av, tb);
      st_col_slot(sX + (size_t)i * 256, v, lane);
      st_c(a.Xi + ((size_t)i * nb + j) * 256, v, lane);
    }
    __syncthreads();
  }
}

// ---- kernel U: K^-1 = L^-T L^-1, one lower block per workgroup ----------------
// Z_ij = sum_{k >= i} X_ki^T X_kj (i >= j); diagonal blocks made exactly
// symmetric.
__global__ __launch_bounds__(64) void nll_lauum_kernel(NllArgs a) {
  __shared__ double sT[256];
  if (a.out[1] != 1.0) return;
  const int nb = a.nb, lane = threadIdx.x;
  int I = 0, J = 0;
  advance_lower(I, J, blockIdx.x);
  d4_t Zv = zero4();
  for (int k = I; k < nb; k += 4) {
    double av[4][4], bv[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (k + u < nb) {
        ld_cols(a.Xi + ((size_t)(k + u) * nb + I) * 256, lane, av[u]);  // X_ki^T as an A operand
        ld_cols(a.Xi + ((size_t)(k + u) * nb + J) * 256, lane, bv[u]);  // X_kj as a B operand
      }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (k + u < nb) Zv = mma16(Zv, av[u], bv[u]);
  }
  if (I == J) {
    const int g = lane >> 4, c = lane & 15;
    st_c(sT, Zv, lane);
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 4; ++r) Zv[r] = 0.5 * (Zv[r] + sT[c * 16 + g + 4 * r]);
  }
  st_c(a.Z + ((size_t)I * nb + J) * 256, Zv, lane);
}

// ---- kernel V: alpha = K^-1 r and r^T alpha per block of 16 rows --------------
__global__ __launch_bounds__(64) void nll_alpha_kernel(NllArgs a) {
  if (a.out[1] != 1.0) return;
  const int nb = a.nb, I = blockIdx.x, lane = threadIdx.x;
  const int rowoff = (lane & 15) * 16 + (lane >> 4);
  double acc = 0.0;
  for (int J = 0; J < nb; J += 4) {
    double av[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int JJ = J + u;
      if (JJ < nb) {
        const bool below = JJ < I;  // Z_IJ stored, else Z_JI^T (Z_II is symmetric)
        const double* p = a.Z + (below ? (size_t)I * nb + JJ : (size_t)JJ * nb + I) * 256 + (below ? rowoff : lane);
        const int str = below ? 4 : 64;
#pragma unroll
        for (int s = 0; s < 4; ++s) av[u][s] = p[s * str];
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (J + u < nb)
#pragma unroll
        for (int s = 0; s < 4; ++s) acc += av[u][s] * a.r[16 * (J + u) + 4 * s + (lane >> 4)];
  }
  acc += __shfl_xor(acc, 16);
  acc += __shfl_xor(acc, 32);
  double q = 0.0;
  if (lane < 16) {
    a.alpha[16 * I + lane] = acc;
    q = acc * a.r[16 * I + lane];
  }
  q = wave_sum(q);
  if (lane == 0) a.qpart[I] = q;
}

// ---- kernel B: gradient partial sums ----------------------------------------
template <int D, bool LW>
__global__ __launch_bounds__(kGradThreads) void nll_grad_kernel(NllArgs a) {
  constexpr int P = LW ? 3 * D + 2 : D + 2;
  __shared__ double sRed[kGradThreads / 64][P];
  if (a.out[1] != 1.0) return;  // K not positive definite: no gradient
  const int nb = a.nb, m = a.m, t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const bool m52 = a.m52 != 0;
  const double s2 = exp(a.theta[D]), tau2 = exp(a.theta[D + 1]);
  const double root = m52 ? kRoot5 : kRoot3;
  double inv_ls[D];
#pragma unroll
  for (int k = 0; k < D; ++k) inv_ls[k] = exp(-a.theta[k]);
  const double* X = LW ? a.Xw : a.X;
  double g[P];
#pragma unroll
  for (int p = 0; p < P; ++p) g[p] = 0.0;
  const int n_lower = nb * (nb + 1) / 2;
  int I = 0, J = 0;
  advance_lower(I, J, blockIdx.x);
  for (int b = blockIdx.x; b < n_lower; b += gridDim.x, advance_lower(I, J, gridDim.x)) {
    const int ii = t >> 4, jj = t & 15, i = 16 * I + ii, j = 16 * J + jj;
    if ((I == J && jj > ii) || i >= m || j >= m) continue;
    const double zij = a.Z[((size_t)I * nb + J) * 256 + t];
    const double w = 0.5 * (i == j ? 1.0 : 2.0) * (a.alpha[i] * a.alpha[j] - zij);  // W and dK are symmetric
    double tk[D], r2 = 0.0;
#pragma unroll
    for (int k = 0; k < D; ++k) {
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
    for (int w = 0; w < kGradThreads / 64; ++w) s += sRed[w][t];
    a.part[(size_t)blockIdx.x * P + t] = s;
  }
}

// ---- kernel C: the NLL, and the gradient's partial sums in block order -------
// Workgroup p < P adds parameter p's kGradBlocks partial sums (one per lane,
// a fixed butterfly); workgroup P forms the NLL from the quadratic form's
// per-block parts and the pivots' products.
__global__ __launch_bounds__(64) void nll_finish_kernel(NllArgs a, int P, int with_grad) {
  if (a.out[1] != 1.0) return;
  const int lane = threadIdx.x, p = blockIdx.x;
  if (p < P) {
    if (!with_grad) return;
    const double v = wave_sum(lane < kGradBlocks ? a.part[(size_t)lane * P + p] : 0.0);
    if (lane == 0) a.out[2 + p] = v;
  } else if (lane == 0) {
    double q = 0.0, logdet = 0.0;
    for (int k = 0; k < a.nb; ++k) {
      q += a.qpart[k];
      logdet += log(a.prod[k]);
    }
    a.out[0] = 0.5 * q + 0.5 * logdet + 0.5 * a.m * kLog2PiD;
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
    const size_t n = up(md) + up(mp) + 3 * blocks + (size_t)nb_ * 256 + (learn_warp ? 3 * up(md) : 0) + up(mp) +
                     2 * up(nb_) +
                     up(2 + P_) + up((size_t)kGradBlocks * P_);
    if (hipMalloc(&buf_, n * sizeof(double)) != hipSuccess) {
      buf_ = nullptr;
      return fail(SCOOT_ERR_NO_MEMORY, "gp nll: device allocation failed");
    }
    if (hipHostMalloc(&host_, (2 + P_) * sizeof(double), hipHostMallocDefault) != hipSuccess) {
      host_ = nullptr;
      return fail(SCOOT_ERR_NO_MEMORY, "gp nll: pinned allocation failed");
    }
    double* p = buf_;
    double* Xd = p;
    p += up(md);
    double* rd = p;
    p += up(mp);
    a_.L = p;
    p += blocks;
    a_.Z = p;
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
    a_.prod = p;
    p += up(nb_);
    a_.qpart = p;
    p += up(nb_);
    a_.out = p;
    p += up(2 + P_);
    a_.part = p;
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
    lds_ = ((size_t)nb_ * 256 + 16 * 17 + 16 + 256 + SCOOT_MAX_OBS / 16 + kNllWaves + 2 + kNllWaves) * sizeof(double);
    lds_tri_ = ((size_t)nb_ + kTriWaves) * 256 * sizeof(double);
    const int rc = allow_full_lds((const void*)nll_factor_kernel, "gp nll");
    return rc != SCOOT_OK ? rc : allow_full_lds((const void*)nll_trtri_kernel, "gp nll");
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
    hipLaunchKernelGGL(nll_trtri_kernel, dim3((unsigned)nb_), dim3(kTriWaves * 64), lds_tri_, s_, a_);
    hipLaunchKernelGGL(nll_lauum_kernel, dim3((unsigned)(nb_ * (nb_ + 1) / 2)), dim3(64), 0, s_, a_);
    hipLaunchKernelGGL(nll_alpha_kernel, dim3((unsigned)nb_), dim3(64), 0, s_, a_);
    if (grad) {
      const int rc = by_dim<1>(d_, [&](auto D) {
        if (lw_)
          hipLaunchKernelGGL((nll_grad_kernel<decltype(D)::value, true>), dim3(kGradBlocks), dim3(kGradThreads), 0,
                             s_, a_);
        else
          hipLaunchKernelGGL((nll_grad_kernel<decltype(D)::value, false>), dim3(kGradBlocks), dim3(kGradThreads), 0,
                             s_, a_);
        return SCOOT_OK;
      });
      if (rc != SCOOT_OK) {
        rc_ = rc;
        return false;
      }
    }
    hipLaunchKernelGGL(nll_finish_kernel, dim3((unsigned)(P_ + 1)), dim3(64), 0, s_, a_, P_, grad ? 1 : 0);
    const hipError_t launched = hipGetLastError();
    if (launched != hipSuccess) {
      rc_ = fail(SCOOT_ERR_DEVICE, std::string("gp nll: launch failed: ") + hipGetErrorString(launched));
      return false;
    }
    if (hipMemcpyAsync(host_, a_.out, (2 + P_) * sizeof(double), hipMemcpyDeviceToHost, s_) != hipSuccess ||
        hipStreamSynchronize(s_) != hipSuccess) {
      rc_ = fail(SCOOT_ERR_DEVICE, std::string("gp nll: device evaluation failed: ") +
                                       hipGetErrorString(hipGetLastError()));
      return false;
    }
    if (host_[1] != 1.0) return false;
    *nll = host_[0];
    if (grad) std::memcpy(grad, host_ + 2, sizeof(double) * P_);
    return true;
  }
  int error() const { return rc_; }

 private:
  hipStream_t s_ = nullptr;
  int m_ = 0, d_ = 0, nb_ = 0, P_ = 0;
  bool lw_ = false;
  size_t lds_ = 0, lds_tri_ = 0;
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

}  // namespace scoot
