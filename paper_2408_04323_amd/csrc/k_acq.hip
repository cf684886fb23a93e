// Acquisition kernels: EI (Sec. 4.4.1, Eq. 8) and EHVI (Sec. 4.4.2, Eq. 9),
// objectives minimised.
//
// Both rest on the partial expectation G(c) = E[(c - Y)^+], Y ~ N(mu, sd^2):
//   G(c) = sd * h(u),  u = (c - mu) / sd,  h(u) = u Phi(u) + phi(u),
// and G(c) = max(0, c - mu) when sd = 0 (normal.h evaluates it).
//
// EI  = G(best + xi).
// EHVI = sum over boxes B = [l, u] of prod_j (G_j(u_j) - G_j(l_j)), G_j(-inf) = 0,
// with the boxes and their coordinates built on the host.
// * one or two objectives: the boxes are the column strips of the front in
//   order of the first objective, [a_i, a_{i+1}] x [-inf, h_i]; each thread
//   streams them, G_1 at consecutive a's carried in a register, no tables;
// * three objectives: the boxes are columns [a_i, a_{i+1}] of the first axis,
//   each cut along the second axis into consecutive ranges [b_j, b_k] over
//   which the open region is [-inf, h] on the third.  Per column the EHVI
//   term is (G_0(a_{i+1}) - G_0(a_i)) * sum over its boxes of
//   (G_1(b_k) - G_1(b_j)) * G_2(h): each thread tabulates G_1 and G_2 at
//   their axes' coordinates in its own LDS column, evaluates G_0 once per
//   column, carries G_1 from one box to the next (the ranges are
//   consecutive), so a box costs two table reads, a subtraction and an fma;
//   the box records (k, h) arrive through wave-uniform loads.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "internal.h"
#include "normal.h"
#include "select.h"

namespace scoot {

template <typename T>
__global__ __launch_bounds__(256) void ei_kernel(const T* __restrict__ mu, const T* __restrict__ sd,
                                                 int64_t n, T c, T* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const T si = sd[i];
    out[i] = partial_expectation<T>(c, mu[i], si, reciprocal(si));
  }
}

constexpr int kEhviThreads = 64;
constexpr int kStripThreads = 256;

// p <= 2: boxes in strip order; hi holds, per box, a_{i+1} (axis 0) and
// h_i (axis 1, unused when p = 1); a_0 = -inf.  The table is read with
// wave-uniform indices: either from device memory (a pointer) or, when it
// fits, straight from the kernel arguments (StripArgTable), which spares an
// upload before every launch.
constexpr int kStripArgBytes = 2048;
template <typename T>
struct StripArgTable {
  T v[kStripArgBytes / sizeof(T)];
  __device__ T operator[](int i) const { return v[i]; }
};
// EHVI of one candidate over the strips: G_0 at consecutive a's carried.
template <typename T, int P, typename Table>
__device__ inline T strip_ehvi(const Table& hi, int n_boxes, T m0, T s0, T m1, T s1) {
  const T r0 = reciprocal(s0);
  const T r1 = P == 2 ? reciprocal(s1) : T(0);
  T g_prev = T(0), acc = T(0);
  for (int b = 0; b < n_boxes; ++b) {
    const T g_next = partial_expectation<T>(hi[2 * b], m0, s0, r0);
    const T w = P == 2 ? partial_expectation<T>(hi[2 * b + 1], m1, s1, r1) : T(1);
    acc += (g_next - g_prev) * w;
    g_prev = g_next;
  }
  return acc;
}

template <typename T, int P, typename Table>
__global__ __launch_bounds__(kStripThreads) void ehvi_strip_kernel(const T* __restrict__ mu0, const T* __restrict__ mu1,
                                                                   const T* __restrict__ sd0, const T* __restrict__ sd1,
                                                                   const Table hi, int n_boxes, int64_t n,
                                                                   T* __restrict__ out) {
  for (int64_t c = (int64_t)blockIdx.x * kStripThreads + threadIdx.x; c < n; c += (int64_t)gridDim.x * kStripThreads) {
    const T m0 = mu0[c], s0 = sd0[c];
    const T m1 = P == 2 ? mu1[c] : T(0), s1 = P == 2 ? sd1[c] : T(0);
    out[c] = strip_ehvi<T, P>(hi, n_boxes, m0, s0, m1, s1);
  }
}

// The same EHVI with the first stage of the top-q selection (Sec. 4.6) in its
// epilogue, so that the scores are not read back: every candidate's score and
// mask byte form its key in registers (select.h), each wave keeps a running
// best-q list over its chunks of 64 candidates (a chunk enters the list only
// when some key beats the list's q-th entry), and at the end the workgroup's
// sixteen lists are merged into one: part_keys [grid x q] and part_count
// [grid] (eligible candidates) go to stage 2.  The EHVI scores are still
// written.  Workgroups of sixteen waves keep the lists stage 2 reads few
// (n / 1024 x q) while every wave still scores a single chunk of 64 at the
// pool sizes of the workloads, as in the plain EHVI kernel.
constexpr int kStripSelThreads = 1024;
constexpr int kStripSelWaves = kStripSelThreads / 64;

template <typename T, typename K, int P, typename Table>
__global__ __launch_bounds__(kStripSelThreads) void ehvi_strip_select_kernel(
    const T* __restrict__ mu0, const T* __restrict__ mu1, const T* __restrict__ sd0, const T* __restrict__ sd1,
    const Table hi, int n_boxes, int64_t n, T* __restrict__ out, const uint8_t* __restrict__ mask, int q,
    K* __restrict__ part_keys, int32_t* __restrict__ part_count) {
  __shared__ K wave_lists[kStripSelWaves * SCOOT_MAX_Q];
  __shared__ int32_t wave_valid[kStripSelWaves];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  K list{};
  int32_t valid = 0;
  for (int64_t base = ((int64_t)blockIdx.x * kStripSelWaves + wave) * 64; base < n;
       base += (int64_t)gridDim.x * kStripSelThreads) {
    const int64_t c = base + lane;
    const bool live = c < n;
    const int64_t ci = live ? c : n - 1;
    const T m0 = mu0[ci], s0 = sd0[ci];
    const T m1 = P == 2 ? mu1[ci] : T(0), s1 = P == 2 ? sd1[ci] : T(0);
    const uint8_t ok = mask ? mask[ci] : (uint8_t)1;
    const T acc = strip_ehvi<T, P>(hi, n_boxes, m0, s0, m1, s1);
    if (live) out[c] = acc;
    const K key = make_key(acc, c, live && ok != 0);
    valid += key.zero() ? 0 : 1;
    if (__any(key > list_entry(list, q - 1))) {
      K keys[1] = {key};
      wave_select<K, 1>(keys, list, q);
    }
  }
  for (int m = 32; m >= 1; m >>= 1) valid += __shfl_xor(valid, m);
  if (lane < q) wave_lists[wave * q + lane] = list;
  if (lane == 0) wave_valid[wave] = valid;
  __syncthreads();
  if (wave != 0) return;
  K keys[kStripSelWaves];  // kStripSelWaves x q <= kStripSelWaves x 64 entries
#pragma unroll
  for (int j = 0; j < kStripSelWaves; ++j) {
    const int i = j * 64 + lane;
    keys[j] = i < kStripSelWaves * q ? wave_lists[i] : K{};
  }
  K merged{};
  wave_select<K, kStripSelWaves>(keys, merged, q);
  if (lane < q) part_keys[(int64_t)blockIdx.x * q + lane] = merged;
  if (lane == 0) {
    int32_t sum = 0;
#pragma unroll
    for (int w = 0; w < kStripSelWaves; ++w) sum += wave_valid[w];
    part_count[blockIdx.x] = sum;
  }
}

// Three objectives.  coords: axis 0 (n0 values), then axis 1 (n1), then
// axis 2 (n2), each starting at -inf.  rec[b] = k | (n1 + h) << 16: the LDS
// rows of G_1(b_k) and G_2(c_h) for box b; col_end[i] = one past the last box
// of column i (i = 0 .. n0 - 2); the boxes of a column start at j = 0.  The
// records arrive through wave-uniform (scalar) loads, four boxes per load in
// the unrolled loop.
struct Ehvi3Args {
  int64_t n;
  int n0, n1, n2;
};

template <typename T>
__global__ __launch_bounds__(kEhviThreads) void ehvi3_kernel(
    const T* __restrict__ mu0, const T* __restrict__ mu1, const T* __restrict__ mu2,
    const T* __restrict__ sd0, const T* __restrict__ sd1, const T* __restrict__ sd2,
    const T* __restrict__ coords, const uint32_t* __restrict__ rec, const uint32_t* __restrict__ col_end,
    T* __restrict__ out, const Ehvi3Args a) {
  extern __shared__ __align__(16) unsigned char smem[];
  T* g = reinterpret_cast<T*>(smem);  // [n1 + n2][kEhviThreads]: G_1 then G_2
  const int tid = threadIdx.x;
  int64_t c = (int64_t)blockIdx.x * kEhviThreads + tid;
  const bool live = c < a.n;
  if (!live) c = a.n - 1;
  const T m0 = mu0[c], s0 = sd0[c], r0 = reciprocal(s0);
  const T m1 = mu1[c], s1 = sd1[c], r1 = reciprocal(s1);
  const T m2 = mu2[c], s2 = sd2[c], r2 = reciprocal(s2);
  const T* c0 = coords;
  const T* c1 = coords + a.n0;
  const T* c2 = c1 + a.n1;
  g[tid] = T(0);  // -inf
  for (int q = 1; q < a.n1; ++q) g[q * kEhviThreads + tid] = partial_expectation<T>(c1[q], m1, s1, r1);
  g[a.n1 * kEhviThreads + tid] = T(0);
  for (int q = 1; q < a.n2; ++q)
    g[(a.n1 + q) * kEhviThreads + tid] = partial_expectation<T>(c2[q], m2, s2, r2);
  // Each thread reads only its own column: no barrier needed.
  T acc = T(0), g0_prev = T(0);
  int b = 0;
  for (int i = 0; i + 1 < a.n0; ++i) {
    const T g0 = partial_expectation<T>(c0[i + 1], m0, s0, r0);
    const int end = (int)col_end[i];
    T col = T(0), g1_prev = T(0);
#pragma unroll 4
    for (; b < end; ++b) {
      const uint32_t r = rec[b];
      const T g1 = g[(r & 0xFFFFu) * kEhviThreads + tid];
      const T g2 = g[(r >> 16) * kEhviThreads + tid];
      col += (g1 - g1_prev) * g2;
      g1_prev = g1;
    }
    acc += (g0 - g0_prev) * col;
    g0_prev = g0;
  }
  if (live) out[c] = acc;
}

int launch_ei(const void* mu, const void* sigma, int64_t n, scoot_dtype dt, double c, void* ei,
              void* stream) {
  if (n == 0) return SCOOT_OK;
  hipStream_t s = (hipStream_t)stream;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (dt == SCOOT_F32)
    hipLaunchKernelGGL(ei_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, s, (const float*)mu,
                       (const float*)sigma, n, (float)c, (float*)ei);
  else
    hipLaunchKernelGGL(ei_kernel<double>, dim3((unsigned)blocks), dim3(256), 0, s, (const double*)mu,
                       (const double*)sigma, n, c, (double*)ei);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("ei launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}

namespace {
// Where the fused selection writes (null: EHVI alone).
struct StripSelect {
  const uint8_t* mask;
  int q;
  void* part_keys;
  int32_t* part_count;
  int blocks;
};

template <typename T, int P, typename Table>
void launch_strip(const T* m0, const T* m1, const T* s0, const T* s1, const Table& tab, int nbx, int64_t n, T* out,
                  const StripSelect* sel, int64_t blocks, hipStream_t s) {
  typedef typename std::conditional<std::is_same<T, float>::value, Key64, Key128>::type K;
  if (sel)
    hipLaunchKernelGGL((ehvi_strip_select_kernel<T, K, P, Table>), dim3((unsigned)sel->blocks),
                       dim3(kStripSelThreads), 0, s, m0, m1, s0, s1, tab, nbx, n, out, sel->mask, sel->q,
                       (K*)sel->part_keys, sel->part_count);
  else
    hipLaunchKernelGGL((ehvi_strip_kernel<T, P, Table>), dim3((unsigned)blocks), dim3(kStripThreads), 0, s, m0, m1,
                       s0, s1, tab, nbx, n, out);
}

// One or two objectives: per-box upper coordinates (a_{i+1}, h_i) in strip order.
template <typename T>
int run_ehvi_strip(const void* const* mu, const void* const* sigma, int p, int64_t n, const BoxTable& bt, void* out,
                   hipStream_t s, const StripSelect* sel = nullptr) {
  const int nbx = bt.n_boxes();
  std::vector<T> hi((size_t)nbx * 2, T(0));
  for (int b = 0; b < nbx; ++b) {
    hi[2 * b] = (T)bt.coord[0][bt.hi[(size_t)b * p]];
    if (p == 2) hi[2 * b + 1] = (T)bt.coord[1][bt.hi[(size_t)b * p + 1]];
  }
  int64_t blocks = (n + kStripThreads - 1) / kStripThreads;
  if (blocks > 8192) blocks = 8192;
  const T* m0 = (const T*)mu[0];
  const T* s0 = (const T*)sigma[0];
  const T* m1 = (const T*)(p == 2 ? mu[1] : mu[0]);
  const T* s1 = (const T*)(p == 2 ? sigma[1] : sigma[0]);
  if (hi.size() * sizeof(T) <= kStripArgBytes) {
    StripArgTable<T> tab{};
    std::copy(hi.begin(), hi.end(), tab.v);
    if (p == 2)
      launch_strip<T, 2>(m0, m1, s0, s1, tab, nbx, n, (T*)out, sel, blocks, s);
    else
      launch_strip<T, 1>(m0, m1, s0, s1, tab, nbx, n, (T*)out, sel, blocks, s);
  } else {
    void* dev = device_scratch(hi.size() * sizeof(T), 1);
    if (!dev) return fail(SCOOT_ERR_NO_MEMORY, "ehvi: device scratch allocation failed");
    int rc = upload_async(dev, hi.data(), hi.size() * sizeof(T), 0, s);
    if (rc != SCOOT_OK) return rc;
    const T* tab = (const T*)dev;
    if (p == 2)
      launch_strip<T, 2>(m0, m1, s0, s1, tab, nbx, n, (T*)out, sel, blocks, s);
    else
      launch_strip<T, 1>(m0, m1, s0, s1, tab, nbx, n, (T*)out, sel, blocks, s);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("ehvi launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}

template <typename T>
int run_ehvi3(const void* const* mu, const void* const* sigma, int64_t n, const BoxTable& bt, void* out,
              hipStream_t s) {
  Ehvi3Args a{};
  a.n = n;
  a.n0 = (int)bt.coord[0].size();
  a.n1 = (int)bt.coord[1].size();
  a.n2 = (int)bt.coord[2].size();
  const size_t lds = (size_t)(a.n1 + a.n2) * kEhviThreads * sizeof(T);
  if (lds > 160 * 1024 || a.n1 + a.n2 > 0xFFFF)
    return fail(SCOOT_ERR_UNSUPPORTED, "ehvi: front too large for the on-chip tables");
  // Device blob: coordinates (T), box records, column ends (uint32).
  const int nb = bt.n_boxes();
  const int ncol = a.n0 - 1;
  const size_t coord_bytes = ((size_t)(a.n0 + a.n1 + a.n2) * sizeof(T) + 15) / 16 * 16;
  const size_t rec_bytes = ((size_t)nb * 4 + 15) / 16 * 16;
  std::vector<unsigned char> blob(coord_bytes + rec_bytes + (size_t)ncol * 4, 0);
  T* cc = reinterpret_cast<T*>(blob.data());
  for (int j = 0, at = 0; j < 3; ++j)
    for (double v : bt.coord[j]) cc[at++] = (T)v;
  uint32_t* rr = reinterpret_cast<uint32_t*>(blob.data() + coord_bytes);
  uint32_t* ce = reinterpret_cast<uint32_t*>(blob.data() + coord_bytes + rec_bytes);
  // The boxes come column by column, each column's ranges consecutive from
  // j = 0, the last axis from -inf (build_boxes); anything else is refused.
  int col = 0, j_next = 0;
  for (int b = 0; b < nb; ++b) {
    const int16_t* lo = &bt.lo[(size_t)b * 3];
    const int16_t* hi = &bt.hi[(size_t)b * 3];
    if (lo[0] != col) {
      if (lo[0] != col + 1 || j_next != a.n1 - 1) return fail(SCOOT_ERR_DEVICE, "ehvi: unexpected box layout");
      ce[col++] = (uint32_t)b;
      j_next = 0;
    }
    if (hi[0] != lo[0] + 1 || lo[1] != j_next || hi[1] <= lo[1] || lo[2] != 0 || hi[2] < 1 || hi[2] >= a.n2)
      return fail(SCOOT_ERR_DEVICE, "ehvi: unexpected box layout");
    rr[b] = (uint32_t)hi[1] | (uint32_t)(a.n1 + hi[2]) << 16;
    j_next = hi[1];
  }
  if (nb == 0 || col != ncol - 1 || j_next != a.n1 - 1) return fail(SCOOT_ERR_DEVICE, "ehvi: unexpected box layout");
  ce[col] = (uint32_t)nb;
  void* dev = device_scratch(blob.size(), 1);
  if (!dev) return fail(SCOOT_ERR_NO_MEMORY, "ehvi: device scratch allocation failed");
  int rc = upload_async(dev, blob.data(), blob.size(), 0, s);
  if (rc != SCOOT_OK) return rc;
  const T* coords = reinterpret_cast<const T*>(dev);
  const uint32_t* recs = reinterpret_cast<const uint32_t*>((const unsigned char*)dev + coord_bytes);
  const uint32_t* col_end = reinterpret_cast<const uint32_t*>((const unsigned char*)dev + coord_bytes + rec_bytes);
  const unsigned grid = (unsigned)((n + kEhviThreads - 1) / kEhviThreads);
  rc = allow_full_lds((const void*)ehvi3_kernel<T>, "ehvi");
  if (rc != SCOOT_OK) return rc;
  hipLaunchKernelGGL(ehvi3_kernel<T>, dim3(grid), dim3(kEhviThreads), lds, s, (const T*)mu[0], (const T*)mu[1],
                     (const T*)mu[2], (const T*)sigma[0], (const T*)sigma[1], (const T*)sigma[2], coords, recs,
                     col_end, (T*)out, a);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("ehvi launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}
}  // namespace

int launch_ehvi_topq(const void* const* mu, const void* const* sigma, int p, int64_t n, scoot_dtype dt,
                     const BoxTable& bt, void* ehvi, const uint8_t* mask, int q, int64_t* idx, void* score_out,
                     int32_t* n_valid, void* stream) {
  if (p > 2 || n == 0) {
    const int rc = launch_ehvi(mu, sigma, p, n, dt, bt, ehvi, stream);
    if (rc != SCOOT_OK) return rc;
    return launch_topq(ehvi, mask, n, dt, q, idx, score_out, n_valid, stream);
  }
  hipStream_t s = (hipStream_t)stream;
  // One chunk of 64 per wave up to 512 workgroups (larger pools loop), and at
  // most kSelMaxKeys2 keys for stage 2.
  int64_t blocks = (n + kStripSelThreads - 1) / kStripSelThreads;
  blocks = std::max<int64_t>(1, std::min<int64_t>({blocks, 512, kSelMaxKeys2 / q}));
  const size_t ksz = dt == SCOOT_F32 ? sizeof(Key64) : sizeof(Key128);
  const size_t kbytes = ((size_t)blocks * q * ksz + 255) / 256 * 256;
  unsigned char* ws = (unsigned char*)device_scratch(kbytes + (size_t)blocks * 4, 3);
  if (!ws) return fail(SCOOT_ERR_NO_MEMORY, "ehvi: selection scratch allocation failed");
  const StripSelect sel{mask, q, ws, reinterpret_cast<int32_t*>(ws + kbytes), (int)blocks};
  const int rc = dt == SCOOT_F32 ? run_ehvi_strip<float>(mu, sigma, p, n, bt, ehvi, s, &sel)
                                 : run_ehvi_strip<double>(mu, sigma, p, n, bt, ehvi, s, &sel);
  if (rc != SCOOT_OK) return rc;
  return launch_topq_stage2(ehvi, dt, (int)blocks, q, sel.part_keys, sel.part_count, idx, score_out, n_valid, stream);
}

int launch_ehvi(const void* const* mu, const void* const* sigma, int p, int64_t n, scoot_dtype dt,
                const BoxTable& bt, void* ehvi, void* stream) {
  if (n == 0) return SCOOT_OK;
  hipStream_t s = (hipStream_t)stream;
  if (p <= 2)
    return dt == SCOOT_F32 ? run_ehvi_strip<float>(mu, sigma, p, n, bt, ehvi, s)
                           : run_ehvi_strip<double>(mu, sigma, p, n, bt, ehvi, s);
  return dt == SCOOT_F32 ? run_ehvi3<float>(mu, sigma, n, bt, ehvi, s)
                         : run_ehvi3<double>(mu, sigma, n, bt, ehvi, s);
}

}  // namespace scoot
