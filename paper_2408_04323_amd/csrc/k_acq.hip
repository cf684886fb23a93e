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
// * three objectives: each thread tabulates G_j at every coordinate of every
//   axis in its own LDS column, then sums over the box list (wave-uniform
//   loads).
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"
#include "normal.h"

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

struct EhviArgs {
  int64_t n;
  int n_boxes;
  int n_coord[SCOOT_MAX_OBJECTIVES];
  int coord_off[SCOOT_MAX_OBJECTIVES];
};

constexpr int kEhviThreads = 64;
constexpr int kStripThreads = 256;

// p <= 2: boxes in strip order; coords holds, per box, a_{i+1} (axis 0) and
// h_i (axis 1, unused when p = 1); a_0 = -inf.
template <typename T, int P>
__global__ __launch_bounds__(kStripThreads) void ehvi_strip_kernel(const T* __restrict__ mu0, const T* __restrict__ mu1,
                                                                   const T* __restrict__ sd0, const T* __restrict__ sd1,
                                                                   const T* __restrict__ hi, int n_boxes, int64_t n,
                                                                   T* __restrict__ out) {
  for (int64_t c = (int64_t)blockIdx.x * kStripThreads + threadIdx.x; c < n; c += (int64_t)gridDim.x * kStripThreads) {
    const T m0 = mu0[c], s0 = sd0[c], r0 = reciprocal(s0);
    T m1 = T(0), s1 = T(0), r1 = T(0);
    if (P == 2) {
      m1 = mu1[c];
      s1 = sd1[c];
      r1 = reciprocal(s1);
    }
    T g_prev = T(0), acc = T(0);
    for (int b = 0; b < n_boxes; ++b) {
      const T g_next = partial_expectation<T>(hi[2 * b], m0, s0, r0);
      const T w = P == 2 ? partial_expectation<T>(hi[2 * b + 1], m1, s1, r1) : T(1);
      acc += (g_next - g_prev) * w;
      g_prev = g_next;
    }
    out[c] = acc;
  }
}

// boxes: n_boxes records of 2P uint16 (P lower then P upper coordinate indices)
template <typename T, int P>
__global__ __launch_bounds__(kEhviThreads) void ehvi_kernel(
    const T* __restrict__ mu0, const T* __restrict__ mu1, const T* __restrict__ mu2,
    const T* __restrict__ sd0, const T* __restrict__ sd1, const T* __restrict__ sd2,
    const T* __restrict__ coords, const uint16_t* __restrict__ boxes, T* __restrict__ out,
    const EhviArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  T* g = reinterpret_cast<T*>(smem);  // [sum_j n_coord[j]][kEhviThreads]
  const int tid = threadIdx.x;
  int64_t c = (int64_t)blockIdx.x * kEhviThreads + tid;
  const bool live = c < a.n;
  if (!live) c = a.n - 1;
  const T* mus[3] = {mu0, mu1, mu2};
  const T* sds[3] = {sd0, sd1, sd2};
#pragma unroll
  for (int j = 0; j < P; ++j) {
    const T m = mus[j][c], s = sds[j][c], r = reciprocal(s);
    T* gj = g + (size_t)a.coord_off[j] * kEhviThreads;
    gj[tid] = T(0);  // coordinate 0 is -inf
    for (int q = 1; q < a.n_coord[j]; ++q)
      gj[(size_t)q * kEhviThreads + tid] = partial_expectation<T>(coords[a.coord_off[j] + q], m, s, r);
  }
  // Each thread reads only its own column: no barrier needed.
  T acc = T(0);
  for (int b = 0; b < a.n_boxes; ++b) {
    const uint16_t* bx = boxes + (size_t)b * 2 * P;
    T prod = T(1);
#pragma unroll
    for (int j = 0; j < P; ++j) {
      const T* gj = g + (size_t)a.coord_off[j] * kEhviThreads;
      prod *= gj[(size_t)bx[P + j] * kEhviThreads + tid] - gj[(size_t)bx[j] * kEhviThreads + tid];
    }
    acc += prod;
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
// One or two objectives: per-box upper coordinates (a_{i+1}, h_i) in strip order.
template <typename T>
int run_ehvi_strip(const void* const* mu, const void* const* sigma, int p, int64_t n, const BoxTable& bt, void* out,
                   hipStream_t s) {
  const int nbx = bt.n_boxes();
  std::vector<T> hi((size_t)nbx * 2, T(0));
  for (int b = 0; b < nbx; ++b) {
    hi[2 * b] = (T)bt.coord[0][bt.hi[(size_t)b * p]];
    if (p == 2) hi[2 * b + 1] = (T)bt.coord[1][bt.hi[(size_t)b * p + 1]];
  }
  void* dev = device_scratch(hi.size() * sizeof(T), 1);
  if (!dev) return fail(SCOOT_ERR_NO_MEMORY, "ehvi: device scratch allocation failed");
  int rc = upload_async(dev, hi.data(), hi.size() * sizeof(T), 0, s);
  if (rc != SCOOT_OK) return rc;
  int64_t blocks = (n + kStripThreads - 1) / kStripThreads;
  if (blocks > 8192) blocks = 8192;
  const T* m0 = (const T*)mu[0];
  const T* s0 = (const T*)sigma[0];
  const T* m1 = (const T*)(p == 2 ? mu[1] : mu[0]);
  const T* s1 = (const T*)(p == 2 ? sigma[1] : sigma[0]);
  if (p == 2)
    hipLaunchKernelGGL((ehvi_strip_kernel<T, 2>), dim3((unsigned)blocks), dim3(kStripThreads), 0, s, m0, m1, s0, s1,
                       (const T*)dev, nbx, n, (T*)out);
  else
    hipLaunchKernelGGL((ehvi_strip_kernel<T, 1>), dim3((unsigned)blocks), dim3(kStripThreads), 0, s, m0, m1, s0, s1,
                       (const T*)dev, nbx, n, (T*)out);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("ehvi launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}

template <typename T>
int run_ehvi(const void* const* mu, const void* const* sigma, int p, int64_t n, const BoxTable& bt,
             void* out, hipStream_t s) {
  // Device blob: coordinates (T), then box indices (uint16), uploaded through
  // pinned staging on the stream.
  EhviArgs a{};
  a.n = n;
  a.n_boxes = bt.n_boxes();
  int total = 0;
  for (int j = 0; j < p; ++j) {
    a.coord_off[j] = total;
    a.n_coord[j] = (int)bt.coord[j].size();
    total += a.n_coord[j];
  }
  const size_t lds = (size_t)total * kEhviThreads * sizeof(T);
  if (lds > 160 * 1024) return fail(SCOOT_ERR_UNSUPPORTED, "ehvi: front too large for the on-chip tables");
  const size_t coord_bytes = ((size_t)total * sizeof(T) + 15) / 16 * 16;
  const size_t box_bytes = (size_t)a.n_boxes * 2 * p * sizeof(uint16_t);
  std::vector<unsigned char> blob(coord_bytes + box_bytes, 0);
  T* cc = reinterpret_cast<T*>(blob.data());
  for (int j = 0; j < p; ++j)
    for (int q = 0; q < a.n_coord[j]; ++q) cc[a.coord_off[j] + q] = (T)bt.coord[j][q];
  uint16_t* bb = reinterpret_cast<uint16_t*>(blob.data() + coord_bytes);
  for (int b = 0; b < a.n_boxes; ++b)
    for (int j = 0; j < p; ++j) {
      bb[b * 2 * p + j] = (uint16_t)bt.lo[(size_t)b * p + j];
      bb[b * 2 * p + p + j] = (uint16_t)bt.hi[(size_t)b * p + j];
    }
  void* dev = device_scratch(blob.size(), 1);
  if (!dev) return fail(SCOOT_ERR_NO_MEMORY, "ehvi: device scratch allocation failed");
  int rc = upload_async(dev, blob.data(), blob.size(), 0, s);
  if (rc != SCOOT_OK) return rc;
  const T* coords = reinterpret_cast<const T*>(dev);
  const uint16_t* boxes = reinterpret_cast<const uint16_t*>((const unsigned char*)dev + coord_bytes);
  const T* m[3] = {(const T*)mu[0], (const T*)(p > 1 ? mu[1] : mu[0]), (const T*)(p > 2 ? mu[2] : mu[0])};
  const T* sd[3] = {(const T*)sigma[0], (const T*)(p > 1 ? sigma[1] : sigma[0]),
                    (const T*)(p > 2 ? sigma[2] : sigma[0])};
  const unsigned grid = (unsigned)((n + kEhviThreads - 1) / kEhviThreads);
  static bool attr_set[4] = {false, false, false, false};
  auto launch = [&](auto kern) {
    if (!attr_set[p]) {
      (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
      attr_set[p] = true;
    }
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kEhviThreads), lds, s, m[0], m[1], m[2], sd[0], sd[1],
                       sd[2], coords, boxes, (T*)out, a);
  };
  launch(ehvi_kernel<T, 3>);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("ehvi launch: ") + hipGetErrorString(err));
  return SCOOT_OK;
}
}  // namespace

int launch_ehvi(const void* const* mu, const void* const* sigma, int p, int64_t n, scoot_dtype dt,
                const BoxTable& bt, void* ehvi, void* stream) {
  if (n == 0) return SCOOT_OK;
  hipStream_t s = (hipStream_t)stream;
  if (p <= 2)
    return dt == SCOOT_F32 ? run_ehvi_strip<float>(mu, sigma, p, n, bt, ehvi, s)
                           : run_ehvi_strip<double>(mu, sigma, p, n, bt, ehvi, s);
  return dt == SCOOT_F32 ? run_ehvi<float>(mu, sigma, p, n, bt, ehvi, s)
                         : run_ehvi<double>(mu, sigma, p, n, bt, ehvi, s);
}

}  // namespace scoot
