// C ABI of the scoring library: argument checks, handles, library-owned
// scratch, and the order of the device calls.  See include/scoot.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <set>
#include <utility>
#include <string>
#include <vector>

#include "internal.h"

struct scoot_gp_t {
  scoot::GPDevice dev;
  int device = 0;
};
struct scoot_forest_t {
  scoot::ForestDevice dev;
  int device = 0;
};

namespace scoot {

namespace {
thread_local std::string g_last_error;
thread_local const char* g_static_error = nullptr;  // set by fail_static, which allocates nothing

constexpr int kMaxDevices = 64;
constexpr int kScratchSlots = 7;  // used: 1 boxes, 2 votes, 3 top-q, 4 MACE front, 5 warped pool, 6 suggestion step
constexpr int kStagingSlots = 2;

struct Staging {
  void* host = nullptr;
  size_t cap = 0;
  hipEvent_t done = nullptr;
  bool pending = false;
};
struct DeviceState {
  void* scratch[kScratchSlots] = {};
  size_t scratch_cap[kScratchSlots] = {};
  Staging staging[kStagingSlots];
};
std::mutex g_mu;
DeviceState g_dev[kMaxDevices];

int current_device() {
  int d = 0;
  if (hipGetDevice(&d) != hipSuccess) return -1;
  return d;
}
}  // namespace

void clear_error() {
  g_last_error.clear();
  g_static_error = nullptr;
}
void set_error(const std::string& msg) {
  g_static_error = nullptr;
  g_last_error = msg;
}
int fail(int status, const std::string& msg) {
  set_error(msg);
  return status;
}
int fail_static(int status, const char* msg) {
  g_last_error.clear();
  g_static_error = msg;
  return status;
}

void* device_scratch(size_t bytes, int slot) {
  const int d = current_device();
  if (d < 0 || d >= kMaxDevices || slot < 0 || slot >= kScratchSlots) return nullptr;
  std::lock_guard<std::mutex> lk(g_mu);
  DeviceState& st = g_dev[d];
  if (st.scratch_cap[slot] < bytes || !st.scratch[slot]) {
    // Grow-only.  hipFree waits for the device, so work still reading the old
    // buffer has finished before it is released.
    if (st.scratch[slot]) hipFree(st.scratch[slot]);
    st.scratch[slot] = nullptr;
    st.scratch_cap[slot] = 0;
    size_t cap = bytes < 4096 ? 4096 : bytes + bytes / 4;
    if (hipMalloc(&st.scratch[slot], cap) != hipSuccess) {
      st.scratch[slot] = nullptr;
      return nullptr;
    }
    st.scratch_cap[slot] = cap;
  }
  return st.scratch[slot];
}

int allow_full_lds(const void* kernel, const char* what) {
  const int d = current_device();
  if (d < 0) return fail(SCOOT_ERR_DEVICE, std::string(what) + ": no current device");
  std::lock_guard<std::mutex> lk(g_mu);
  static std::set<std::pair<int, const void*>> done;  // (device, kernel) pairs already raised
  if (done.count({d, kernel})) return SCOOT_OK;
  if (hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLdsBytes) != hipSuccess)
    return fail(SCOOT_ERR_DEVICE, std::string(what) + ": cannot raise the kernel's LDS limit");
  done.insert({d, kernel});
  return SCOOT_OK;
}

int upload_async(void* dst, const void* src, size_t bytes, int slot, void* stream) {
  const int d = current_device();
  if (d < 0 || d >= kMaxDevices || slot < 0 || slot >= kStagingSlots)
    return fail(SCOOT_ERR_DEVICE, "upload: no current device");
  if (bytes == 0) return SCOOT_OK;
  std::lock_guard<std::mutex> lk(g_mu);
  Staging& sg = g_dev[d].staging[slot];
  if (sg.pending) {
    if (hipEventSynchronize(sg.done) != hipSuccess) return fail(SCOOT_ERR_DEVICE, "upload: event wait failed");
    sg.pending = false;
  }
  if (!sg.done && hipEventCreateWithFlags(&sg.done, hipEventDisableTiming) != hipSuccess)
    return fail(SCOOT_ERR_DEVICE, "upload: event creation failed");
  if (sg.cap < bytes) {
    if (sg.host) hipHostFree(sg.host);
    sg.host = nullptr;
    sg.cap = 0;
    size_t cap = bytes < 65536 ? 65536 : bytes;
    if (hipHostMalloc(&sg.host, cap, hipHostMallocDefault) != hipSuccess) {
      sg.host = nullptr;
      return fail(SCOOT_ERR_NO_MEMORY, "upload: pinned staging allocation failed");
    }
    sg.cap = cap;
  }
  std::memcpy(sg.host, src, bytes);
  hipStream_t s = (hipStream_t)stream;
  if (hipMemcpyAsync(dst, sg.host, bytes, hipMemcpyHostToDevice, s) != hipSuccess)
    return fail(SCOOT_ERR_DEVICE, "upload: hipMemcpyAsync failed");
  if (hipEventRecord(sg.done, s) != hipSuccess) return fail(SCOOT_ERR_DEVICE, "upload: event record failed");
  sg.pending = true;
  return SCOOT_OK;
}

int gp_from_fit(const FitHost& f, const double* warp_a, const double* warp_b, scoot_dtype dt, scoot_gp* out) {
  const int m = f.m, d = f.d;
  const double signal_var = f.s2, noise_var = f.tau2, prior_mean = f.c;
  try {
    GPDevice g;
    g.dt = dt;
    g.m = m;
    g.d = d;
    g.m_pad = f.m_pad;
    g.nb = f.nb;
    g.s2 = signal_var;
    g.tau2 = noise_var;
    g.c = prior_mean;
    for (int k = 0; k < SCOOT_MAX_DIM; ++k) {
      g.scale64[k] = k < d ? f.scale[k] : 0.0;
      g.scale32[k] = (float)g.scale64[k];
    }
    for (int i = 0; i < 3; ++i) {
      g.coef64[i] = f.coef[i];
      g.coef32[i] = (float)f.coef[i];
    }
    g.warp = warp_a != nullptr;
    for (int k = 0; k < SCOOT_MAX_DIM; ++k) {
      g.warp_a[k] = g.warp && k < d ? warp_a[k] : 1.0;
      g.warp_b[k] = g.warp && k < d ? warp_b[k] : 1.0;
    }

    // Host image of the device buffer: [L^-1 packed][scaled observations][alpha][alpha as float].
    std::vector<unsigned char> img;
    size_t linv_bytes, xs_bytes;
    const size_t esz = dt == SCOOT_F32 ? 4 : 8;
    std::vector<float> l32;
    std::vector<double> l64;
    if (dt == SCOOT_F32) {
      pack_linv_f32(f, l32);
      linv_bytes = l32.size() * 4;
    } else {
      pack_linv_f64(f, l64);
      linv_bytes = l64.size() * 8;
    }
    linv_bytes = (linv_bytes + 255) / 256 * 256;
    // fp32: the augmented observation rows of the cross-term chain (double);
    // fp64: scaled rows of kXsStride doubles
    std::vector<double> q32;
    if (dt == SCOOT_F32) pack_obs_f32(f, q32);
    xs_bytes = dt == SCOOT_F32 ? (q32.size() * 8 + 255) / 256 * 256
                               : ((size_t)f.m_pad * kXsStride * esz + 255) / 256 * 256;
    const size_t alpha_bytes = (size_t)f.m_pad * 8;
    const size_t alpha32_bytes = ((size_t)f.m_pad * 4 + 255) / 256 * 256;
    img.assign(linv_bytes + xs_bytes + alpha_bytes + alpha32_bytes, 0);
    if (dt == SCOOT_F32) std::memcpy(img.data(), l32.data(), l32.size() * 4);
    else std::memcpy(img.data(), l64.data(), l64.size() * 8);
    // fp64 rows with a spare column carry alpha_i in column d, so the kernel
    // reads an observation and its weight with the same loads.
    if (dt == SCOOT_F32) {
      std::memcpy(img.data() + linv_bytes, q32.data(), q32.size() * 8);
    } else {
      for (int i = 0; i < f.m_pad; ++i)
        for (int k = 0; k < kXsStride; ++k) {
          double v = 0.0;
          if (k < d) v = i < m ? f.Xw[(size_t)i * d + k] * f.scale[k] : kPadCoord;
          else if (k == d && i < m) v = f.alpha[i];
          std::memcpy(img.data() + linv_bytes + ((size_t)i * kXsStride + k) * 8, &v, 8);
        }
    }
    std::vector<double> apad(f.m_pad, 0.0);
    std::memcpy(apad.data(), f.alpha.data(), sizeof(double) * m);
    std::memcpy(img.data() + linv_bytes + xs_bytes, apad.data(), alpha_bytes);
    for (int i = 0; i < f.m_pad; ++i) {
      float av = (float)apad[i];
      std::memcpy(img.data() + linv_bytes + xs_bytes + alpha_bytes + (size_t)i * 4, &av, 4);
    }

    hipError_t e = hipMalloc(&g.buf, img.size());
    if (e != hipSuccess) return fail(SCOOT_ERR_NO_MEMORY, "gp fit: device allocation failed");
    e = hipMemcpy(g.buf, img.data(), img.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      hipFree(g.buf);
      return fail(SCOOT_ERR_DEVICE, std::string("gp fit: upload: ") + hipGetErrorString(e));
    }
    g.linv = g.buf;
    g.xs = (unsigned char*)g.buf + linv_bytes;
    g.alpha = (const double*)((unsigned char*)g.buf + linv_bytes + xs_bytes);
    g.alpha32 = (const float*)((unsigned char*)g.buf + linv_bytes + xs_bytes + alpha_bytes);
    scoot_gp h = new scoot_gp_t;
    h->dev = g;
    hipGetDevice(&h->device);
    *out = h;
    return SCOOT_OK;
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "gp fit: host allocation failed");
  }
}

}  // namespace scoot

using namespace scoot;

namespace {
constexpr double kLn2 = 0.69314718055994530942;

bool check_dtype(scoot_dtype dt) { return dt == SCOOT_F32 || dt == SCOOT_F64; }

int device_error(const char* what, hipError_t e) {
  return fail(SCOOT_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}
}  // namespace

extern "C" {

int scoot_abi_version(void) { return SCOOT_ABI_VERSION; }

const char* scoot_status_string(int status) {
  switch (status) {
    case SCOOT_OK: return "ok";
    case SCOOT_ERR_INVALID_ARG: return "invalid argument";
    case SCOOT_ERR_NOT_PD: return "matrix not positive definite";
    case SCOOT_ERR_DEVICE: return "device error";
    case SCOOT_ERR_UNSUPPORTED: return "unsupported size";
    case SCOOT_ERR_NO_MEMORY: return "out of memory";
    default: return "unknown status";
  }
}

const char* scoot_last_error(void) { return g_static_error ? g_static_error : g_last_error.c_str(); }

int scoot_gp_factor_host_ex(const double* X, const double* y, int m, int d, scoot_kernel kernel,
                            const double* lengthscale, const double* warp_a, const double* warp_b,
                            double signal_var, double noise_var, double prior_mean, double* L, double* alpha) {
  clear_error();
  if (!L || !alpha) return fail(SCOOT_ERR_INVALID_ARG, "gp factor: null output");
  try {
    FitHost f;
    int rc = fit_host(X, y, m, d, kernel, lengthscale, warp_a, warp_b, signal_var, noise_var, prior_mean, f);
    if (rc != SCOOT_OK) return rc;
    std::memcpy(L, f.L.data(), sizeof(double) * (size_t)m * m);
    std::memcpy(alpha, f.alpha.data(), sizeof(double) * (size_t)m);
    return SCOOT_OK;
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "gp factor: host allocation failed");
  }
}

int scoot_gp_factor_host(const double* X, const double* y, int m, int d, const double* lengthscale,
                         double signal_var, double noise_var, double prior_mean, double* L, double* alpha) {
  return scoot_gp_factor_host_ex(X, y, m, d, SCOOT_MATERN52, lengthscale, nullptr, nullptr, signal_var, noise_var,
                                 prior_mean, L, alpha);
}

int scoot_gp_fit(const double* X, const double* y, int m, int d, const double* lengthscale, double signal_var,
                 double noise_var, double prior_mean, scoot_dtype dt, void* stream, scoot_gp* out) {
  return scoot_gp_fit_ex(X, y, m, d, SCOOT_MATERN52, lengthscale, nullptr, nullptr, signal_var, noise_var,
                         prior_mean, dt, stream, out);
}

int scoot_gp_fit_ex(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* lengthscale,
                    const double* warp_a, const double* warp_b, double signal_var, double noise_var,
                    double prior_mean, scoot_dtype dt, void* stream, scoot_gp* out) {
  clear_error();
  (void)stream;
  if (!out) return fail(SCOOT_ERR_INVALID_ARG, "gp fit: null output handle");
  *out = nullptr;
  if (!check_dtype(dt)) return fail(SCOOT_ERR_INVALID_ARG, "gp fit: bad dtype");
  try {
    FitHost f;
    int rc = fit_host(X, y, m, d, kernel, lengthscale, warp_a, warp_b, signal_var, noise_var, prior_mean, f);
    if (rc != SCOOT_OK) return rc;
    return gp_from_fit(f, warp_a, warp_b, dt, out);
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "gp fit: host allocation failed");
  }
}

int scoot_gp_fit_device(const double* X, const double* y, int m, int d, scoot_kernel kernel,
                        const double* lengthscale, const double* warp_a, const double* warp_b, double signal_var,
                        double noise_var, double prior_mean, scoot_dtype dt, void* stream, scoot_gp* out) {
  clear_error();
  if (!out) return fail(SCOOT_ERR_INVALID_ARG, "gp fit: null output handle");
  *out = nullptr;
  if (!check_dtype(dt)) return fail(SCOOT_ERR_INVALID_ARG, "gp fit: bad dtype");
  try {
    return gp_fit_device(X, y, m, d, kernel, lengthscale, warp_a, warp_b, signal_var, noise_var, prior_mean, dt,
                         stream, out);
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "gp fit: host allocation failed");
  }
}

int scoot_gp_nll(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                 const double* warp_b, double prior_mean, const double* theta, double* nll, double* grad) {
  clear_error();
  try {
    return mle_nll(X, y, m, d, kernel, warp_a, warp_b, prior_mean, theta, nll, grad);
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "gp nll: host allocation failed");
  }
}

int scoot_gp_mle(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                 const double* warp_b, double prior_mean, const double* lower, const double* upper, int max_iter,
                 double* theta, double* nll, int* iterations) {
  clear_error();
  try {
    return mle_fit(X, y, m, d, kernel, warp_a, warp_b, prior_mean, lower, upper, max_iter, theta, nll, iterations);
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "gp mle: host allocation failed");
  }
}

int scoot_gp_nll_warp(const double* X, const double* y, int m, int d, scoot_kernel kernel, double prior_mean,
                      const double* theta, double* nll, double* grad) {
  clear_error();
  try {
    return mle_nll(X, y, m, d, kernel, nullptr, nullptr, prior_mean, theta, nll, grad, true);
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "gp nll: host allocation failed");
  }
}

int scoot_gp_mle_warp(const double* X, const double* y, int m, int d, scoot_kernel kernel, double prior_mean,
                      const double* lower, const double* upper, int max_iter, double* theta, double* nll,
                      int* iterations) {
  clear_error();
  try {
    return mle_fit(X, y, m, d, kernel, nullptr, nullptr, prior_mean, lower, upper, max_iter, theta, nll, iterations,
                   true);
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "gp mle: host allocation failed");
  }
}

int scoot_gp_nll_device(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                        const double* warp_b, double prior_mean, int learn_warp, const double* theta, double* nll,
                        double* grad, void* stream) {
  clear_error();
  try {
    return mle_nll_device(X, y, m, d, kernel, warp_a, warp_b, prior_mean, learn_warp != 0, theta, nll, grad, stream);
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "gp nll: host allocation failed");
  }
}

int scoot_gp_mle_device(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                        const double* warp_b, double prior_mean, int learn_warp, const double* lower,
                        const double* upper, int max_iter, double* theta, double* nll, int* iterations,
                        void* stream) {
  clear_error();
  try {
    return mle_fit_device(X, y, m, d, kernel, warp_a, warp_b, prior_mean, learn_warp != 0, lower, upper, max_iter,
                          theta, nll, iterations, stream);
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "gp mle: host allocation failed");
  }
}

int scoot_gp_destroy(scoot_gp gp) {
  clear_error();
  if (!gp) return SCOOT_OK;
  if (gp->dev.buf) hipFree(gp->dev.buf);
  delete gp;
  return SCOOT_OK;
}

int scoot_posterior(scoot_gp gp, const float* Xc, int64_t n, void* mu, void* sigma, void* stream) {
  clear_error();
  if (!gp) return fail(SCOOT_ERR_INVALID_ARG, "posterior: null handle");
  if (n < 0) return fail(SCOOT_ERR_INVALID_ARG, "posterior: n < 0");
  if (n > 0 && (!Xc || !mu || !sigma)) return fail(SCOOT_ERR_INVALID_ARG, "posterior: null pointer");
  return launch_posterior(gp->dev, Xc, n, mu, sigma, nullptr, nullptr, stream);
}

int scoot_acq_ei(const void* mu, const void* sigma, int64_t n, scoot_dtype dt, double best_y, double xi,
                 void* ei, void* stream) {
  clear_error();
  if (!check_dtype(dt) || n < 0) return fail(SCOOT_ERR_INVALID_ARG, "ei: bad dtype or n");
  if (n > 0 && (!mu || !sigma || !ei)) return fail(SCOOT_ERR_INVALID_ARG, "ei: null pointer");
  if (!std::isfinite(best_y) || !std::isfinite(xi)) return fail(SCOOT_ERR_INVALID_ARG, "ei: non-finite best_y/xi");
  return launch_ei(mu, sigma, n, dt, best_y + xi, ei, stream);
}

int scoot_ehvi_front(const double* Y_obs, int m_obs, int p, const double* ref, double* front, int* n_front,
                     int* n_boxes) {
  clear_error();
  if (!n_front) return fail(SCOOT_ERR_INVALID_ARG, "ehvi front: null n_front");
  try {
    BoxTable bt;
    int rc = build_boxes(Y_obs, m_obs, p, ref, bt);
    if (rc != SCOOT_OK) return rc;
    *n_front = bt.n_front;
    if (front && bt.n_front) std::memcpy(front, bt.front.data(), sizeof(double) * bt.front.size());
    if (n_boxes) *n_boxes = bt.n_boxes();
    return SCOOT_OK;
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "ehvi front: host allocation failed");
  }
}

int scoot_acq_ehvi(const void* const* mu, const void* const* sigma, int p, int64_t n, scoot_dtype dt,
                   const double* Y_obs, int m_obs, const double* ref, void* ehvi, void* stream) {
  clear_error();
  if (!check_dtype(dt) || n < 0 || p < 1 || p > SCOOT_MAX_OBJECTIVES)
    return fail(SCOOT_ERR_INVALID_ARG, "ehvi: bad dtype, n or p");
  if (n > 0) {
    if (!mu || !sigma || !ehvi) return fail(SCOOT_ERR_INVALID_ARG, "ehvi: null pointer");
    for (int j = 0; j < p; ++j)
      if (!mu[j] || !sigma[j]) return fail(SCOOT_ERR_INVALID_ARG, "ehvi: null objective pointer");
  }
  try {
    BoxTable bt;
    int rc = build_boxes(Y_obs, m_obs, p, ref, bt);
    if (rc != SCOOT_OK) return rc;
    return launch_ehvi(mu, sigma, p, n, dt, bt, ehvi, stream);
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "ehvi: host allocation failed");
  }
}

int scoot_forest_create(const int32_t* feature, const float* threshold, const int32_t* left, const int32_t* right,
                        const int32_t* leaf_q16, const int64_t* tree_offset, int n_trees, int d,
                        scoot_forest* out) {
  clear_error();
  if (!out) return fail(SCOOT_ERR_INVALID_ARG, "forest: null output handle");
  *out = nullptr;
  try {
    ForestHost fh;
    int rc = pack_forest(feature, threshold, left, right, leaf_q16, tree_offset, n_trees, d, fh);
    if (rc != SCOOT_OK) return rc;
    ForestDevice f;
    f.n_trees = n_trees;
    f.d = d;
    f.chunk_tree = fh.chunk_tree;
    f.chunk_first_node = fh.chunk_first_node;
    const size_t nb = fh.nodes.size() * 4, rb = fh.root.size() * 4, db = fh.depth.size() * 4,
                 lb = fh.leaf_orig.size() * 4, tb = fh.tree_orig.size() * 4;
    hipError_t e = hipMalloc(&f.nodes, nb + rb + db + lb + tb);
    if (e != hipSuccess) return fail(SCOOT_ERR_NO_MEMORY, "forest: device allocation failed");
    f.root = (uint32_t*)((unsigned char*)f.nodes + nb);
    f.depth = (uint32_t*)((unsigned char*)f.root + rb);
    f.leaf_orig = (int32_t*)((unsigned char*)f.depth + db);
    f.tree_orig = (int32_t*)((unsigned char*)f.leaf_orig + lb);
    e = hipMemcpy(f.nodes, fh.nodes.data(), nb, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(f.root, fh.root.data(), rb, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(f.depth, fh.depth.data(), db, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(f.leaf_orig, fh.leaf_orig.data(), lb, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(f.tree_orig, fh.tree_orig.data(), tb, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      hipFree(f.nodes);
      return device_error("forest: upload", e);
    }
    scoot_forest h = new scoot_forest_t;
    h->dev = f;
    hipGetDevice(&h->device);
    *out = h;
    return SCOOT_OK;
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "forest: host allocation failed");
  }
}

int scoot_forest_train(const double* X, const double* y, int n, int d, int n_trees, int max_depth, uint64_t seed,
                       int bootstrap, int64_t capacity, int32_t* feature, double* threshold, int32_t* left,
                       int32_t* right, double* value, int64_t* tree_offset, int64_t* n_nodes) {
  clear_error();
  if (!n_nodes) return fail(SCOOT_ERR_INVALID_ARG, "forest train: null n_nodes");
  try {
    TrainedForest tf;
    int rc = train_forest_host(X, y, n, d, n_trees, max_depth, seed, bootstrap != 0, tf);
    if (rc != SCOOT_OK) return rc;
    const int64_t total = (int64_t)tf.feature.size();
    *n_nodes = total;
    if (!feature) return SCOOT_OK;  // size query
    if (!threshold || !left || !right || !value || !tree_offset)
      return fail(SCOOT_ERR_INVALID_ARG, "forest train: null output array");
    if (capacity < total) return fail(SCOOT_ERR_INVALID_ARG, "forest train: capacity below the node count");
    std::memcpy(feature, tf.feature.data(), sizeof(int32_t) * total);
    std::memcpy(threshold, tf.threshold.data(), sizeof(double) * total);
    std::memcpy(left, tf.left.data(), sizeof(int32_t) * total);
    std::memcpy(right, tf.right.data(), sizeof(int32_t) * total);
    std::memcpy(value, tf.value.data(), sizeof(double) * total);
    std::memcpy(tree_offset, tf.tree_offset.data(), sizeof(int64_t) * (n_trees + 1));
    return SCOOT_OK;
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "forest train: host allocation failed");
  }
}

int scoot_forest_train_create(const double* X, const double* y, int n, int d, int n_trees, int max_depth,
                              uint64_t seed, int bootstrap, scoot_forest* out) {
  clear_error();
  if (!out) return fail(SCOOT_ERR_INVALID_ARG, "forest train: null output handle");
  *out = nullptr;
  try {
    TrainedForest tf;
    int rc = train_forest_host(X, y, n, d, n_trees, max_depth, seed, bootstrap != 0, tf);
    if (rc != SCOOT_OK) return rc;
    // device format: thresholds rounded down to float32 (x <= t keeps its
    // decision for every float32 x), leaf values in Q16 (half to even)
    const size_t total = tf.feature.size();
    std::vector<int32_t> feat(total), q16(total, 0);
    std::vector<float> thr(total, 0.0f);
    for (size_t k = 0; k < total; ++k) {
      const bool leaf = tf.left[k] < 0;
      feat[k] = leaf ? 0 : tf.feature[k];
      if (!leaf) {
        float t32 = (float)tf.threshold[k];
        if ((double)t32 > tf.threshold[k]) t32 = std::nextafter(t32, -INFINITY);
        thr[k] = t32;
      } else {
        q16[k] = (int32_t)std::nearbyint(tf.value[k] * 65536.0);
      }
    }
    return scoot_forest_create(feat.data(), thr.data(), tf.left.data(), tf.right.data(), q16.data(),
                               tf.tree_offset.data(), n_trees, d, out);
  } catch (const std::bad_alloc&) {
    return fail(SCOOT_ERR_NO_MEMORY, "forest train: host allocation failed");
  }
}

int scoot_forest_destroy(scoot_forest f) {
  clear_error();
  if (!f) return SCOOT_OK;
  if (f->dev.nodes) hipFree(f->dev.nodes);
  delete f;
  return SCOOT_OK;
}

int scoot_vote_threshold(double delta, int n_trees, int64_t* votes_min) {
  clear_error();
  if (!votes_min || !(delta >= 0.0 && delta <= 1.0) || n_trees < 1 || n_trees > SCOOT_MAX_TREES)
    return fail(SCOOT_ERR_INVALID_ARG, "vote threshold: delta must be in [0,1], 1 <= T <= SCOOT_MAX_TREES");
  *votes_min = (int64_t)std::ceil(delta * (double)((int64_t)n_trees * 65536));
  return SCOOT_OK;
}

int scoot_rf_feasibility(scoot_forest f, const float* Xc, int64_t n, double delta, int32_t* votes, uint8_t* mask,
                         int32_t* leaf_idx, void* stream) {
  clear_error();
  if (!f) return fail(SCOOT_ERR_INVALID_ARG, "rf: null forest");
  if (n < 0 || (n > 0 && !Xc)) return fail(SCOOT_ERR_INVALID_ARG, "rf: bad n or null pool");
  int64_t vmin = 0;
  int rc = scoot_vote_threshold(delta, f->dev.n_trees, &vmin);
  if (rc != SCOOT_OK) return rc;
  return launch_forest(f->dev, Xc, n, vmin, votes, mask, leaf_idx, stream);
}

int scoot_suggest_topq(const void* score, const uint8_t* mask, int64_t n, scoot_dtype dt, int q, int64_t* idx,
                       void* score_out, int32_t* n_valid, void* stream) {
  clear_error();
  if (!check_dtype(dt)) return fail(SCOOT_ERR_INVALID_ARG, "topq: bad dtype");
  if (q < 1 || q > SCOOT_MAX_Q) return fail(SCOOT_ERR_INVALID_ARG, "topq: q must be in 1..SCOOT_MAX_Q");
  if (n < 0 || n >= ((int64_t)1 << 31)) return fail(SCOOT_ERR_INVALID_ARG, "topq: n out of range");
  if (!idx || (n > 0 && !score)) return fail(SCOOT_ERR_INVALID_ARG, "topq: null pointer");
  return launch_topq(score, mask, n, dt, q, idx, score_out, n_valid, stream);
}

int scoot_suggest_topq_noalloc(const void* score, const uint8_t* mask, int64_t n, scoot_dtype dt, int q, int64_t* idx,
                               void* score_out, int32_t* n_valid, void* stream) {
  clear_error();
  if (!check_dtype(dt)) return fail_static(SCOOT_ERR_INVALID_ARG, "topq (no allocation): bad dtype");
  if (q < 1 || q > SCOOT_MAX_Q)
    return fail_static(SCOOT_ERR_INVALID_ARG, "topq (no allocation): q must be in 1..SCOOT_MAX_Q");
  if (n < 0 || n >= ((int64_t)1 << 31)) return fail_static(SCOOT_ERR_INVALID_ARG, "topq (no allocation): n out of range");
  if (!idx || (n > 0 && !score)) return fail_static(SCOOT_ERR_INVALID_ARG, "topq (no allocation): null pointer");
  return launch_topq_static(score, mask, n, dt, q, idx, score_out, n_valid, stream);
}

int scoot_ucb_beta(int t, double* beta) {
  clear_error();
  if (!beta || t < 1) return fail(SCOOT_ERR_INVALID_ARG, "ucb beta: null beta or t < 1");
  const double tt = (double)t, delta = 1.0 / (tt * tt), pi = 3.14159265358979323846;
  *beta = 2.0 * std::log(tt * tt * pi * pi / (6.0 * delta));
  return SCOOT_OK;
}

int scoot_acq_mace(const void* mu, const void* sigma, int64_t n, scoot_dtype dt, double best_y, double xi, double beta,
                   void* ucb, void* pi, void* ei, void* stream) {
  clear_error();
  if (!check_dtype(dt) || n < 0) return fail(SCOOT_ERR_INVALID_ARG, "mace: bad dtype or n");
  if (n > 0 && (!mu || !sigma || !ucb || !pi || !ei)) return fail(SCOOT_ERR_INVALID_ARG, "mace: null pointer");
  if (!std::isfinite(best_y) || !std::isfinite(xi) || !std::isfinite(beta))
    return fail(SCOOT_ERR_INVALID_ARG, "mace: non-finite best_y/xi/beta");
  return launch_mace_scores(mu, sigma, n, dt, best_y + xi, beta, ucb, pi, ei, stream);
}

int scoot_pareto_front3(const void* a, const void* b, const void* c, const uint8_t* mask, int64_t n, scoot_dtype dt,
                        uint8_t* front, int32_t* n_front, void* stream) {
  clear_error();
  if (!check_dtype(dt)) return fail(SCOOT_ERR_INVALID_ARG, "pareto: bad dtype");
  if (n < 0 || n >= ((int64_t)1 << 31)) return fail(SCOOT_ERR_INVALID_ARG, "pareto: n out of range");
  if (n > 0 && (!a || !b || !c || !front)) return fail(SCOOT_ERR_INVALID_ARG, "pareto: null pointer");
  return launch_pareto_front3(a, b, c, mask, n, dt, front, n_front, stream);
}

int scoot_random_pick(const uint8_t* flags, int64_t n, uint64_t seed, int q, int64_t* idx, int32_t* n_flagged,
                      void* stream) {
  clear_error();
  if (q < 1 || q > SCOOT_MAX_Q) return fail(SCOOT_ERR_INVALID_ARG, "pick: q must be in 1..SCOOT_MAX_Q");
  if (n < 0 || n >= ((int64_t)1 << 31)) return fail(SCOOT_ERR_INVALID_ARG, "pick: n out of range");
  if (!idx || (n > 0 && !flags)) return fail(SCOOT_ERR_INVALID_ARG, "pick: null pointer");
  return launch_random_pick(flags, n, seed, q, idx, n_flagged, stream);
}

int scoot_suggest_mace(scoot_gp gp, scoot_forest f, const float* Xc, int64_t n, double best_y, double xi, double beta,
                       double delta, uint64_t seed, int q, void* mu, void* sigma, void* ucb, void* pi, void* ei,
                       int32_t* votes, uint8_t* mask, uint8_t* front, int64_t* idx, int32_t* n_front, void* stream) {
  return scoot_suggest_mace_ex(gp, f, nullptr, Xc, n, best_y, xi, beta, delta, seed, q, mu, sigma, ucb, pi, ei, votes,
                               mask, front, idx, n_front, stream);
}

int scoot_suggest_mace_ex(scoot_gp gp, scoot_forest f, const uint8_t* known, const float* Xc, int64_t n,
                          double best_y, double xi, double beta, double delta, uint64_t seed, int q, void* mu,
                          void* sigma, void* ucb, void* pi, void* ei, int32_t* votes, uint8_t* mask, uint8_t* front,
                          int64_t* idx, int32_t* n_front, void* stream) {
  clear_error();
  if (!gp) return fail(SCOOT_ERR_INVALID_ARG, "mace suggest: null GP");
  if (n < 0 || n >= ((int64_t)1 << 31)) return fail(SCOOT_ERR_INVALID_ARG, "mace suggest: n out of range");
  if (n > 0 && (!Xc || !mu || !sigma || !ucb || !pi || !ei || !mask || !front))
    return fail(SCOOT_ERR_INVALID_ARG, "mace suggest: null pointer");
  if (!idx) return fail(SCOOT_ERR_INVALID_ARG, "mace suggest: null idx");
  if (q < 1 || q > SCOOT_MAX_Q) return fail(SCOOT_ERR_INVALID_ARG, "mace suggest: q out of range");
  if (!std::isfinite(best_y) || !std::isfinite(xi) || !std::isfinite(beta))
    return fail(SCOOT_ERR_INVALID_ARG, "mace suggest: non-finite best_y/xi/beta");
  const scoot_dtype dt = gp->dev.dt;
  int64_t vmin = 0;
  int rc;
  if (f) {
    rc = scoot_vote_threshold(delta, f->dev.n_trees, &vmin);
    if (rc != SCOOT_OK) return rc;
  }
  rc = launch_posterior(gp->dev, Xc, n, mu, sigma, nullptr, nullptr, stream);
  if (rc != SCOOT_OK) return rc;
  rc = launch_mace_scores(mu, sigma, n, dt, best_y + xi, beta, ucb, pi, ei, stream);
  if (rc != SCOOT_OK) return rc;
  rc = f ? launch_forest(f->dev, Xc, n, vmin, votes, mask, nullptr, stream, known)
         : launch_mask_init(mask, known, n, stream);
  if (rc != SCOOT_OK) return rc;
  rc = launch_pareto_front3(ucb, pi, ei, mask, n, dt, front, nullptr, stream);
  if (rc != SCOOT_OK) return rc;
  return launch_random_pick(front, n, seed, q, idx, n_front, stream);
}

int scoot_sobol_pool(const uint32_t* poly, const uint32_t* vinit, int d, const int32_t* levels, int64_t skip, int64_t n,
                     const double* A, const double* b, int r, float* Xc, uint8_t* known, void* stream) {
  clear_error();
  return launch_sobol_pool(poly, vinit, d, levels, skip, n, A, b, r, Xc, known, stream);
}

int scoot_known_constraints(const float* Xc, int64_t n, int d, const double* A, const double* b, int r,
                            uint8_t* known, void* stream) {
  clear_error();
  return launch_known_constraints(Xc, n, d, A, b, r, known, stream);
}

int scoot_delta_update(double* delta, int* c, int k, int any_invalid) {
  clear_error();
  if (!delta || !c || k < 0) return fail(SCOOT_ERR_INVALID_ARG, "delta update: null pointer or k < 0");
  if (any_invalid) {
    double v = *delta + 0.05;
    if (v < 0.5) v = 0.5;
    if (v > 0.75) v = 0.75;
    *delta = v;
    *c = 0;
  } else {
    *c += k;
    if (*c >= 5) {
      double v = *delta - 0.05;
      *delta = v < 0.25 ? 0.25 : v;
      *c -= 5;
    }
  }
  return SCOOT_OK;
}

int scoot_score_pool(const scoot_gp* gps, int p, scoot_forest f, const float* Xc, int64_t n, double best_y,
                     double xi, const double* Y_obs, int m_obs, const double* ref, double delta, int q, void* mu,
                     void* sigma, void* acq, int32_t* votes, uint8_t* mask, int64_t* idx, void* score_out,
                     int32_t* n_valid, void* stream) {
  return scoot_score_pool_ex(gps, p, f, nullptr, Xc, n, best_y, xi, Y_obs, m_obs, ref, delta, q, mu, sigma, acq, votes,
                             mask, idx, score_out, n_valid, stream);
}

int scoot_score_pool_ex(const scoot_gp* gps, int p, scoot_forest f, const uint8_t* known, const float* Xc, int64_t n,
                        double best_y, double xi, const double* Y_obs, int m_obs, const double* ref, double delta,
                        int q, void* mu, void* sigma, void* acq, int32_t* votes, uint8_t* mask, int64_t* idx,
                        void* score_out, int32_t* n_valid, void* stream) {
  clear_error();
  if (!gps || p < 1 || p > SCOOT_MAX_OBJECTIVES) return fail(SCOOT_ERR_INVALID_ARG, "score pool: bad p or gps");
  for (int j = 0; j < p; ++j)
    if (!gps[j] || gps[j]->dev.dt != gps[0]->dev.dt || gps[j]->dev.d != gps[0]->dev.d)
      return fail(SCOOT_ERR_INVALID_ARG, "score pool: GPs must share dtype and d");
  if (n < 0 || n >= ((int64_t)1 << 31)) return fail(SCOOT_ERR_INVALID_ARG, "score pool: n out of range");
  if (n > 0 && (!Xc || !mu || !sigma || !acq || !mask)) return fail(SCOOT_ERR_INVALID_ARG, "score pool: null pointer");
  if (!idx) return fail(SCOOT_ERR_INVALID_ARG, "score pool: null idx");
  if (q < 1 || q > SCOOT_MAX_Q) return fail(SCOOT_ERR_INVALID_ARG, "score pool: q out of range");
  const scoot_dtype dt = gps[0]->dev.dt;
  const size_t esz = dt == SCOOT_F32 ? 4 : 8;
  const void* mus[SCOOT_MAX_OBJECTIVES];
  const void* sds[SCOOT_MAX_OBJECTIVES];
  int rc;
  BoxTable bt;
  if (p > 1) {
    try {
      rc = build_boxes(Y_obs, m_obs, p, ref, bt);
    } catch (const std::bad_alloc&) {
      return fail(SCOOT_ERR_NO_MEMORY, "score pool: host allocation failed");
    }
    if (rc != SCOOT_OK) return rc;
  } else if (!std::isfinite(best_y) || !std::isfinite(xi)) {
    return fail(SCOOT_ERR_INVALID_ARG, "score pool: non-finite best_y/xi");
  }
  int64_t vmin = 0;
  if (f) {
    rc = scoot_vote_threshold(delta, f->dev.n_trees, &vmin);
    if (rc != SCOOT_OK) return rc;
  }
  // The mask first, so that the selection can run in the acquisition's epilogue.
  rc = f ? launch_forest(f->dev, Xc, n, vmin, votes, mask, nullptr, stream, known)
         : launch_mask_init(mask, known, n, stream);
  if (rc != SCOOT_OK) return rc;
  for (int j = 0; j < p; ++j) {
    void* mj = (unsigned char*)mu + (size_t)j * n * esz;
    void* sj = (unsigned char*)sigma + (size_t)j * n * esz;
    mus[j] = mj;
    sds[j] = sj;
    if (p == 1) {
      const double c = best_y + xi;
      rc = launch_posterior(gps[j]->dev, Xc, n, mj, sj, &c, acq, stream);
    } else {
      rc = launch_posterior(gps[j]->dev, Xc, n, mj, sj, nullptr, nullptr, stream);
    }
    if (rc != SCOOT_OK) return rc;
  }
  if (p > 1) return launch_ehvi_topq(mus, sds, p, n, dt, bt, acq, mask, q, idx, score_out, n_valid, stream);
  return launch_topq(acq, mask, n, dt, q, idx, score_out, n_valid, stream);
}

namespace {
int kb_check(const scoot_gp* gps, int p, int64_t n, int q, const GPDevice** g) {
  if (!gps || p < 1 || p > SCOOT_MAX_OBJECTIVES) return fail(SCOOT_ERR_INVALID_ARG, "believer: bad p or gps");
  if (n < 1 || n >= ((int64_t)1 << 31) || q < 1 || q > SCOOT_MAX_Q)
    return fail(SCOOT_ERR_INVALID_ARG, "believer: bad n or q");
  for (int j = 0; j < p; ++j) {
    if (!gps[j]) return fail(SCOOT_ERR_INVALID_ARG, "believer: null GP");
    if (gps[j]->dev.dt != SCOOT_F32) return fail(SCOOT_ERR_UNSUPPORTED, "believer: float32 GPs only");
    if (gps[j]->dev.d != gps[0]->dev.d) return fail(SCOOT_ERR_INVALID_ARG, "believer: GPs must share d");
    g[j] = &gps[j]->dev;
  }
  return SCOOT_OK;
}
}  // namespace

int scoot_suggest_kb_workspace(const scoot_gp* gps, int p, int64_t n, int q, uint64_t* bytes) {
  clear_error();
  const GPDevice* g[SCOOT_MAX_OBJECTIVES];
  if (!bytes) return fail(SCOOT_ERR_INVALID_ARG, "believer: null bytes");
  int rc = kb_check(gps, p, n, q, g);
  if (rc != SCOOT_OK) return rc;
  *bytes = kb_workspace_bytes(g, p, n, q);
  return SCOOT_OK;
}

int scoot_suggest_kb(const scoot_gp* gps, int p, scoot_forest f, const float* Xc, int64_t n, const double* Y_obs,
                     int m_obs, const double* ref, double delta, int q, void* workspace, uint64_t workspace_bytes,
                     int64_t* picks, double* pick_acq, int* n_picked, void* stream) {
  return scoot_suggest_kb_ex(gps, p, f, nullptr, Xc, n, Y_obs, m_obs, ref, delta, q, workspace, workspace_bytes, picks,
                             pick_acq, n_picked, nullptr, nullptr, stream);
}

int scoot_suggest_kb_ex(const scoot_gp* gps, int p, scoot_forest f, const uint8_t* known, const float* Xc, int64_t n,
                        const double* Y_obs, int m_obs, const double* ref, double delta, int q, void* workspace,
                        uint64_t workspace_bytes, int64_t* picks, double* pick_acq, int* n_picked, float* mu_out,
                        float* sigma_out, void* stream) {
  clear_error();
  const GPDevice* g[SCOOT_MAX_OBJECTIVES];
  int rc = kb_check(gps, p, n, q, g);
  if (rc != SCOOT_OK) return rc;
  if (!Xc || !picks || !n_picked || !ref || (m_obs > 0 && !Y_obs) || m_obs < 0)
    return fail(SCOOT_ERR_INVALID_ARG, "believer: null pointer");
  int64_t vmin = 0;
  if (f) {
    rc = scoot_vote_threshold(delta, f->dev.n_trees, &vmin);
    if (rc != SCOOT_OK) return rc;
  }
  const size_t need = kb_workspace_bytes(g, p, n, q);
  void* ws = workspace;
  bool own = false;
  if (!ws) {
    if (hipMalloc(&ws, need) != hipSuccess) return fail(SCOOT_ERR_NO_MEMORY, "believer: workspace allocation failed");
    own = true;
  } else if (workspace_bytes < need) {
    return fail(SCOOT_ERR_INVALID_ARG, "believer: workspace too small");
  }
  try {
    rc = run_kriging_believer(g, p, f ? &f->dev : nullptr, known, vmin, Xc, n, Y_obs, m_obs, ref, q, ws, picks, pick_acq,
                              n_picked, mu_out, sigma_out, stream);
  } catch (const std::bad_alloc&) {
    rc = fail(SCOOT_ERR_NO_MEMORY, "believer: host allocation failed");
  }
  if (own) {
    (void)hipStreamSynchronize((hipStream_t)stream);
    (void)hipFree(ws);
  }
  return rc;
}

}  // extern "C"
