// Candidate generation on the device: a Sobol pool on the search space's
// grids, and the known-constraint mask (Sec. 4.5.3: the optimiser's space is
// pruned by constraints known beforehand; Sec. 4.7: missing suggestions are
// filled with Sobol points; Sec. 4.1 and Algorithm 1: the first observations
// are Sobol points; the engines' rules are listed in the appendix on known
// constraints).
//
// Sobol points (Sobol 1967, direction numbers by the recurrence of Bratley and
// Fox 1988, Gray-code order of Antonov and Saleev 1979): coordinate j of point
// i is the XOR of V_j[k] over the set bits k of gray(i) = i ^ (i >> 1), over
// 2^32.  Consecutive points differ by one direction number: point i + 1 is
// point i XOR V_j[ctz(i + 1)].  A thread owns one dimension of a run of 16
// points whose first index is a multiple of 16, so inside the run the
// direction numbers it needs are V_j[0..3] in a fixed order; only the run's
// first point is built bit by bit.  The block's points are staged row-major
// in LDS and leave in coalesced stores; the known-constraint rows are
// evaluated on the staged float32 values in the same pass.
//
// Grids: level count L >= 2 rounds u to rint(u (L - 1)) / (L - 1) in double
// (half to even), L = 1 is a boolean (1 when u >= 1/2), L = 0 is continuous;
// the result is stored as float32.  A candidate is admissible when every
// constraint row sum_k A[r][k] x_k <= b[r] holds, the sum taken over k in
// order in double with each product and each sum rounded separately.  Linear
// rows express every rule the paper lists: an order between two knobs, two
// switches that exclude each other, one switch that requires another, and a
// bound that applies unless a boolean is set (big-M on the boolean).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <string>

#include "internal.h"

namespace scoot {

namespace {

constexpr int kSobolThreads = 256;
constexpr int kSobolRun = 16;       // points per thread; runs start at multiples of 16
constexpr int kSobolBits = 32;

struct Constraints {
  double A[SCOOT_MAX_CONSTRAINTS * SCOOT_MAX_DIM];  // row-major r x d
  double b[SCOOT_MAX_CONSTRAINTS];
  int r, d;
};

struct SobolArgs {
  uint32_t v[kSobolBits * SCOOT_MAX_DIM];  // [k][j]: direction number k of dimension j (k-major, stride d)
  int32_t levels[SCOOT_MAX_DIM];
  Constraints con;
  int64_t n;
  int64_t row0;   // pool row of the first run's first point: -(skip mod 16)
  uint64_t first; // Sobol index of that point: skip - (skip mod 16)
  int nbits;      // bit length of the last index generated
  int runs_per_block;
};
static_assert(sizeof(SobolArgs) <= 4096, "kernel arguments are limited to 4 KiB");

__device__ inline float snap_level(uint32_t x, int L) {
  if (L == 0) return (float)x * 0x1p-32f;  // x -> float rounds to nearest; the scaling is exact
  if (L == 1) return x >= 0x80000000u ? 1.0f : 0.0f;
  const double q = (double)(L - 1);
  return (float)(rint((double)x * 0x1p-32 * q) / q);
}

// Sequential, separately rounded row sums (no fused multiply-add).
__device__ inline bool admissible(const float* x, int stride, const Constraints& c) {
#pragma clang fp contract(off)
  bool ok = true;
  for (int r = 0; r < c.r; ++r) {
    double s = 0.0;
    for (int k = 0; k < c.d; ++k) s = s + c.A[r * c.d + k] * (double)x[k * stride];
    ok = ok && s <= c.b[r];
  }
  return ok;
}

__global__ __launch_bounds__(kSobolThreads) void sobol_pool_kernel(float* __restrict__ Xc, uint8_t* __restrict__ known,
                                                                   const SobolArgs a) {
  __shared__ uint32_t vs[kSobolBits * SCOOT_MAX_DIM];
  __shared__ float tile[kSobolThreads * kSobolRun];  // runs_per_block * 16 points x d, row-major
  const int tid = threadIdx.x, d = a.con.d, R = a.runs_per_block;
  for (int i = tid; i < kSobolBits * d; i += kSobolThreads) vs[i] = a.v[i];
  __syncthreads();

  const int run = tid / d, j = tid - run * d;
  if (run < R) {
    const uint64_t i0 = a.first + ((uint64_t)blockIdx.x * R + run) * kSobolRun;
    const uint64_t g = i0 ^ (i0 >> 1);
    uint32_t x = 0;
    for (int k = 0; k < a.nbits; ++k) x ^= vs[k * d + j] & (0u - (uint32_t)((g >> k) & 1u));
    const uint32_t v0 = vs[j], v1 = vs[d + j], v2 = vs[2 * d + j], v3 = vs[3 * d + j];
    const int L = a.levels[j];
    float* out = tile + run * kSobolRun * d + j;
#pragma unroll
    for (int t = 0; t < kSobolRun; ++t) {
      out[t * d] = snap_level(x, L);
      if (t + 1 < kSobolRun) {
        const int c = __builtin_ctz(t + 1);  // 0..3, fixed at compile time
        x ^= c == 0 ? v0 : c == 1 ? v1 : c == 2 ? v2 : v3;
      }
    }
  }
  __syncthreads();

  const int pts = R * kSobolRun;
  const int64_t row_base = a.row0 + (int64_t)blockIdx.x * pts;
  const int64_t e_base = row_base * d, e_end = a.n * d;
  for (int e = tid; e < pts * d; e += kSobolThreads) {
    const int64_t ge = e_base + e;
    if (ge >= 0 && ge < e_end) Xc[ge] = tile[e];
  }
  if (known) {
    for (int p = tid; p < pts; p += kSobolThreads) {
      const int64_t row = row_base + p;
      if (row >= 0 && row < a.n) known[row] = admissible(tile + p * d, 1, a.con) ? 1 : 0;
    }
  }
}

__global__ __launch_bounds__(256) void known_constraints_kernel(const float* __restrict__ Xc, int64_t n,
                                                                uint8_t* __restrict__ known, const Constraints c) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    known[i] = admissible(Xc + i * c.d, 1, c) ? 1 : 0;
}

__global__ void mask_init_kernel(uint8_t* __restrict__ mask, const uint8_t* __restrict__ known, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    mask[i] = known ? (known[i] != 0 ? 1 : 0) : 1;
}

int check_constraints(const double* A, const double* b, int r, int d, Constraints& c) {
  if (r < 0 || r > SCOOT_MAX_CONSTRAINTS)
    return fail(SCOOT_ERR_UNSUPPORTED, "known constraints: r must be in 0..SCOOT_MAX_CONSTRAINTS");
  if (r > 0 && (!A || !b)) return fail(SCOOT_ERR_INVALID_ARG, "known constraints: null A or b");
  std::memset(&c, 0, sizeof(c));
  c.r = r;
  c.d = d;
  for (int i = 0; i < r * d; ++i) {
    if (!std::isfinite(A[i])) return fail(SCOOT_ERR_INVALID_ARG, "known constraints: non-finite A");
    c.A[i] = A[i];
  }
  for (int i = 0; i < r; ++i) {
    if (std::isnan(b[i])) return fail(SCOOT_ERR_INVALID_ARG, "known constraints: NaN b");
    c.b[i] = b[i];
  }
  return SCOOT_OK;
}

// Direction numbers V[k] = m_k 2^(32 - k), k = 1..32, of the dimension with
// primitive polynomial `poly` (bit t = coefficient of x^t; degree s = its bit
// length - 1) and initial values m_1..m_s.  Beyond s, m_k is the XOR of
// 2^t a_t m_(k-t) over t = 1..s-1 (a_t the coefficient of x^(s-t)) with
// m_(k-s) and 2^s m_(k-s).
int direction_numbers(uint32_t poly, const uint32_t* vinit, uint32_t* V) {
  if (poly == 0 || (poly & 1u) == 0) return fail(SCOOT_ERR_INVALID_ARG, "sobol: polynomial must have constant term 1");
  int s = 31;
  while (!((poly >> s) & 1u)) --s;
  if (s > SCOOT_SOBOL_MAX_DEGREE) return fail(SCOOT_ERR_UNSUPPORTED, "sobol: polynomial degree above SCOOT_SOBOL_MAX_DEGREE");
  uint64_t m[kSobolBits + 1];
  for (int k = 1; k <= kSobolBits; ++k) {
    if (s == 0) {
      m[k] = 1;
    } else if (k <= s) {
      m[k] = vinit[k - 1];
      if ((m[k] & 1u) == 0 || m[k] >= ((uint64_t)1 << k))
        return fail(SCOOT_ERR_INVALID_ARG, "sobol: initial value m_k must be odd and below 2^k");
    } else {
      uint64_t v = m[k - s] ^ (m[k - s] << s);
      for (int t = 1; t < s; ++t)
        if ((poly >> (s - t)) & 1u) v ^= m[k - t] << t;
      m[k] = v;
    }
  }
  for (int k = 1; k <= kSobolBits; ++k) V[k - 1] = (uint32_t)(m[k] << (kSobolBits - k));
  return SCOOT_OK;
}

int launched(const char* what) {
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(err));
  return SCOOT_OK;
}

}  // namespace

int launch_sobol_pool(const uint32_t* poly, const uint32_t* vinit, int d, const int32_t* levels, int64_t skip,
                      int64_t n, const double* A, const double* b, int r, float* Xc, uint8_t* known, void* stream) {
  if (d < 1 || d > SCOOT_MAX_DIM) return fail(SCOOT_ERR_INVALID_ARG, "sobol: d must be in 1..SCOOT_MAX_DIM");
  if (!poly || !vinit || !levels) return fail(SCOOT_ERR_INVALID_ARG, "sobol: null poly, vinit or levels");
  if (n < 0 || skip < 0 || skip + n > ((int64_t)1 << 32))
    return fail(SCOOT_ERR_INVALID_ARG, "sobol: need n >= 0, skip >= 0, skip + n <= 2^32");
  if (n > 0 && !Xc) return fail(SCOOT_ERR_INVALID_ARG, "sobol: null Xc");
  SobolArgs a;
  std::memset(&a, 0, sizeof(a));
  int rc = check_constraints(A, b, r, d, a.con);
  if (rc != SCOOT_OK) return rc;
  for (int j = 0; j < d; ++j) {
    if (levels[j] < 0) return fail(SCOOT_ERR_INVALID_ARG, "sobol: negative level count");
    a.levels[j] = levels[j];
    uint32_t V[kSobolBits];
    rc = direction_numbers(poly[j], vinit + (size_t)j * SCOOT_SOBOL_MAX_DEGREE, V);
    if (rc != SCOOT_OK) return rc;
    for (int k = 0; k < kSobolBits; ++k) a.v[k * d + j] = V[k];
  }
  if (n == 0) return SCOOT_OK;
  const uint64_t last = (uint64_t)(skip + n - 1);
  a.nbits = 1;
  while (a.nbits < kSobolBits && (last >> a.nbits) != 0) ++a.nbits;
  a.n = n;
  a.row0 = -(skip & (kSobolRun - 1));
  a.first = (uint64_t)skip - (uint64_t)(skip & (kSobolRun - 1));
  a.runs_per_block = kSobolThreads / d;
  const int64_t runs = (n - a.row0 + kSobolRun - 1) / kSobolRun;
  const int64_t blocks = (runs + a.runs_per_block - 1) / a.runs_per_block;
  hipLaunchKernelGGL(sobol_pool_kernel, dim3((unsigned)blocks), dim3(kSobolThreads), 0, (hipStream_t)stream, Xc, known,
                     a);
  return launched("sobol launch");
}

int launch_known_constraints(const float* Xc, int64_t n, int d, const double* A, const double* b, int r,
                             uint8_t* known, void* stream) {
  if (d < 1 || d > SCOOT_MAX_DIM) return fail(SCOOT_ERR_INVALID_ARG, "known constraints: d must be in 1..SCOOT_MAX_DIM");
  if (n < 0 || (n > 0 && (!Xc || !known))) return fail(SCOOT_ERR_INVALID_ARG, "known constraints: bad n or null pointer");
  Constraints c;
  int rc = check_constraints(A, b, r, d, c);
  if (rc != SCOOT_OK) return rc;
  if (n == 0) return SCOOT_OK;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(known_constraints_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, Xc, n, known,
                     c);
  return launched("known constraints launch");
}

int launch_mask_init(uint8_t* mask, const uint8_t* known, int64_t n, void* stream) {
  if (n == 0) return SCOOT_OK;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(mask_init_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, mask, known, n);
  return launched("mask launch");
}

}  // namespace scoot
