// Sequential Kriging-believer selection of q candidates, an extension of the
// parallel suggestion of Sec. 4.6 (the paper takes the top k by EHVI at once).
//
// Each pick x_p joins the observations with the fantasy value y = mu(x_p) and
// the observation noise tau^2.  For a GP with V = L^-1 K*^T kept in memory:
//   L gains the row [v_p^T  d],  v_p = V[:, p],  d = sqrt(sigma^2(x_p) + tau^2),
//   V gains the row v_new(x) = (k(x, x_p) - v_p^T V[:, x]) / d,
//   sigma^2(x) -= v_new(x)^2,  and mu does not move (the fantasy equals it).
// The front gains mu(x_p) of every objective; EHVI is then re-scored over the
// whole pool and the next pick is the top-1 of the feasible, not yet picked
// candidates.  The V row update reads all of V: it is bound by HBM bandwidth.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "internal.h"

namespace scoot {

constexpr int kKbThreads = 256;

// v_p = V[:, pick] (rows entries), and 1 / d with d^2 = sigma(pick)^2 + tau^2.
__global__ __launch_bounds__(kKbThreads) void kb_gather_kernel(const float* __restrict__ V, int64_t ld, int rows,
                                                               int64_t pick, const float* __restrict__ sd, double tau2,
                                                               float* __restrict__ vp, float* __restrict__ dinv) {
  for (int i = threadIdx.x; i < rows; i += kKbThreads) vp[i] = V[(int64_t)i * ld + pick];
  if (threadIdx.x == 0) {
    const double s = (double)sd[pick];
    dinv[0] = (float)(1.0 / sqrt(s * s + tau2));
  }
}

struct KbArgs {
  int64_t n, ld, pick;
  int rows, d;
  float scale[SCOOT_MAX_DIM];
  float c0, c1, c2;
};

// New row of V and the variance downdate, one candidate per thread: each
// thread reads its column of V sixteen rows at a time with every load issued
// before the first is used (a wave keeps 16 x 256 bytes in flight), on two
// accumulation chains.  Measured at n = 2^20, m = 512 against four rows in
// flight: 2% less time per suggestion; two or four candidates per thread
// (8- or 16-byte loads, fewer waves) were slower.  The loads are marked
// non-temporal: V (gigabytes) is streamed once per pick and would only evict
// what the caches hold (3% less time per suggestion at n = 2^20, m = 512).
constexpr int kKbRows = 16;

__global__ __launch_bounds__(kKbThreads) void kb_update_kernel(float* __restrict__ V, const float* __restrict__ vp_g,
                                                               const float* __restrict__ dinv_g,
                                                               const float* __restrict__ Xc, float* __restrict__ sd,
                                                               const KbArgs a) {
  __shared__ float vp[SCOOT_MAX_OBS + SCOOT_MAX_Q + 32];
  for (int i = threadIdx.x; i < a.rows; i += kKbThreads) vp[i] = vp_g[i];
  __syncthreads();
  const float dinv = dinv_g[0];
  const float* xp = Xc + a.pick * a.d;
  for (int64_t x = (int64_t)blockIdx.x * kKbThreads + threadIdx.x; x < a.n; x += (int64_t)gridDim.x * kKbThreads) {
    const float* col = V + x;
    float acc0 = 0.0f, acc1 = 0.0f;
    int i = 0;
    for (; i + kKbRows - 1 < a.rows; i += kKbRows) {
      float v[kKbRows];
#pragma unroll
      for (int r = 0; r < kKbRows; ++r) v[r] = __builtin_nontemporal_load(&col[(int64_t)(i + r) * a.ld]);
#pragma unroll
      for (int r = 0; r < kKbRows; r += 2) {
        acc0 = fmaf(vp[i + r], v[r], acc0);
        acc1 = fmaf(vp[i + r + 1], v[r + 1], acc1);
      }
    }
    for (; i < a.rows; ++i) acc0 = fmaf(vp[i], col[(int64_t)i * a.ld], acc0);
    const float dot = acc0 + acc1;
    // k(x, x_p): same covariance and constants as the posterior kernel
    float r2 = 0.0f;
    for (int k = 0; k < a.d; ++k) {
      const float t = (Xc[x * a.d + k] - xp[k]) * a.scale[k];
      r2 = fmaf(t, t, r2);
    }
    const float u = __builtin_amdgcn_sqrtf(r2);
    const float kxp = fmaf(u, fmaf(u, a.c2, a.c1), a.c0) * __builtin_amdgcn_exp2f(-u);
    const float vnew = (kxp - dot) * dinv;
    V[(int64_t)a.rows * a.ld + x] = vnew;
    const float s = sd[x];
    sd[x] = sqrtf(fmaxf(fmaf(-vnew, vnew, s * s), 0.0f));
  }
}

__global__ void kb_exclude_kernel(uint8_t* __restrict__ eligible, int64_t pick) { eligible[pick] = 0; }

// What the host needs after a top-1, in one place: out = (score, mu_0(pick),
// ..., mu_{p-1}(pick)); the means are left alone when there is no pick.
__global__ void kb_pick_kernel(const int64_t* __restrict__ idx, const float* __restrict__ score,
                               const float* __restrict__ mu, int64_t n, int p, float* __restrict__ out) {
  const int j = threadIdx.x;
  const int64_t pick = idx[0];
  if (j == 0) out[0] = score[0];
  if (j < p && pick >= 0) out[1 + j] = mu[(int64_t)j * n + pick];
}

namespace {
size_t align256(size_t b) { return (b + 255) / 256 * 256; }
// Row stride of a kept V: n rounded up to 64 floats (256 bytes).
int64_t kb_ld(int64_t n) { return (n + 63) / 64 * 64; }

struct KbLayout {
  size_t v, mu, sd, acq, elig, votes, idx, score, nvalid, vp, dinv, pickinfo, xw, total;
};

KbLayout kb_layout(const GPDevice* const* g, int p, int64_t n, int q) {
  KbLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += align256(bytes);
    return at;
  };
  size_t vbytes = 0;
  int rows_max = 0;
  for (int j = 0; j < p; ++j) {
    vbytes += align256((size_t)(g[j]->m_pad + q) * kb_ld(n) * 4);
    rows_max = std::max(rows_max, g[j]->m_pad + q);
  }
  L.v = take(vbytes);
  L.mu = take((size_t)p * n * 4);
  L.sd = take((size_t)p * n * 4);
  L.acq = take((size_t)n * 4);
  L.elig = take((size_t)n);
  L.votes = take((size_t)n * 4);
  L.idx = take(8);
  L.score = take(8);
  L.nvalid = take(4);
  L.vp = take((size_t)p * rows_max * 4);
  L.dinv = take((size_t)p * 4);
  L.pickinfo = take((size_t)(1 + SCOOT_MAX_OBJECTIVES) * 4);
  size_t xw = 0;  // the pool after each warped GP's input warping
  for (int j = 0; j < p; ++j) xw += g[j]->warp ? align256((size_t)n * g[j]->d * 4) : 0;
  L.xw = take(xw);
  L.total = off;
  return L;
}
}  // namespace

size_t kb_workspace_bytes(const GPDevice* const* g, int p, int64_t n, int q) { return kb_layout(g, p, n, q).total; }

int run_kriging_believer(const GPDevice* const* g, int p, const ForestDevice* f, const uint8_t* known,
                         int64_t vote_min, const float* Xc, int64_t n, const double* Y_obs, int m_obs,
                         const double* ref, int q, void* ws, int64_t* picks, double* pick_acq, int* n_picked,
                         float* mu_out, float* sigma_out, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const KbLayout L = kb_layout(g, p, n, q);
  unsigned char* w = (unsigned char*)ws;
  float* V[SCOOT_MAX_OBJECTIVES];
  const int64_t ld = kb_ld(n);
  size_t voff = L.v;
  for (int j = 0; j < p; ++j) {
    V[j] = (float*)(w + voff);
    voff += align256((size_t)(g[j]->m_pad + q) * ld * 4);
  }
  float* mu = (float*)(w + L.mu);
  float* sd = (float*)(w + L.sd);
  float* acq = (float*)(w + L.acq);
  uint8_t* elig = (uint8_t*)(w + L.elig);
  int32_t* votes = (int32_t*)(w + L.votes);
  int64_t* idx = (int64_t*)(w + L.idx);
  float* score = (float*)(w + L.score);
  int32_t* nvalid = (int32_t*)(w + L.nvalid);
  float* vp = (float*)(w + L.vp);
  float* dinv = (float*)(w + L.dinv);
  float* pickinfo = (float*)(w + L.pickinfo);
  int rows_max = 0;
  for (int j = 0; j < p; ++j) rows_max = std::max(rows_max, g[j]->m_pad + q);
  // candidates as each GP sees them: warped copies kept for the whole loop
  const float* xg[SCOOT_MAX_OBJECTIVES];
  size_t xoff = L.xw;
  for (int j = 0; j < p; ++j) {
    xg[j] = Xc;
    if (g[j]->warp) {
      float* xw = (float*)(w + xoff);
      xoff += align256((size_t)n * g[j]->d * 4);
      int rc = launch_warp_pool(*g[j], Xc, n, xw, stream);
      if (rc != SCOOT_OK) return rc;
      xg[j] = xw;
    }
  }

  // Posterior of every objective, V kept; the feasibility mask is the initial eligibility.
  const void* mus[SCOOT_MAX_OBJECTIVES];
  const void* sds[SCOOT_MAX_OBJECTIVES];
  for (int j = 0; j < p; ++j) {
    mus[j] = mu + (size_t)j * n;
    sds[j] = sd + (size_t)j * n;
    int rc = launch_posterior(*g[j], xg[j], n, mu + (size_t)j * n, sd + (size_t)j * n, nullptr, nullptr, stream, V[j],
                              true, ld);
    if (rc != SCOOT_OK) return rc;
  }
  int rc = f ? launch_forest(*f, Xc, n, vote_min, votes, elig, nullptr, stream, known)
             : launch_mask_init(elig, known, n, stream);
  if (rc != SCOOT_OK) return rc;

  std::vector<double> Yaug(Y_obs, Y_obs + (size_t)m_obs * p);
  *n_picked = 0;
  for (int k = 0; k < q; ++k) {
    BoxTable bt;
    rc = build_boxes(Yaug.data(), (int)(Yaug.size() / p), p, ref, bt);
    if (rc != SCOOT_OK) return rc;
    rc = launch_ehvi_topq(mus, sds, p, n, SCOOT_F32, bt, acq, elig, 1, idx, score, nvalid, stream);
    if (rc != SCOOT_OK) return rc;
    // One read-back per pick: the index, its score and its means (the
    // fantasies).  The row updates below are left running while the host
    // builds the next front.
    hipLaunchKernelGGL(kb_pick_kernel, dim3(1), dim3(64), 0, s, idx, score, mu, n, p, pickinfo);
    int64_t pick = -1;
    float info[1 + SCOOT_MAX_OBJECTIVES] = {};
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) e = hipMemcpyAsync(&pick, idx, 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(info, pickinfo, (size_t)(1 + p) * 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("believer: ") + hipGetErrorString(e));
    if (pick < 0) break;
    picks[k] = pick;
    if (pick_acq) pick_acq[k] = info[0];
    *n_picked = k + 1;
    if (k + 1 == q) break;
    // fantasies for the front, then the bordered update of every objective
    for (int j = 0; j < p; ++j) Yaug.push_back((double)info[1 + j]);
    for (int j = 0; j < p; ++j) {
      const int rows = g[j]->m_pad + k;
      float* vpj = vp + (size_t)j * rows_max;
      hipLaunchKernelGGL(kb_gather_kernel, dim3(1), dim3(kKbThreads), 0, s, V[j], ld, rows, pick,
                         sd + (size_t)j * n, g[j]->tau2, vpj, dinv + j);
      KbArgs a{};
      a.n = n;
      a.ld = ld;
      a.pick = pick;
      a.rows = rows;
      a.d = g[j]->d;
      for (int t = 0; t < SCOOT_MAX_DIM; ++t) a.scale[t] = g[j]->scale32[t];
      a.c0 = g[j]->coef32[0];
      a.c1 = g[j]->coef32[1];
      a.c2 = g[j]->coef32[2];
      int64_t blocks = (n + kKbThreads - 1) / kKbThreads;
      if (blocks > 8192) blocks = 8192;
      hipLaunchKernelGGL(kb_update_kernel, dim3((unsigned)blocks), dim3(kKbThreads), 0, s, V[j], vpj, dinv + j, xg[j],
                         sd + (size_t)j * n, a);
    }
    hipLaunchKernelGGL(kb_exclude_kernel, dim3(1), dim3(1), 0, s, elig, pick);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("believer: ") + hipGetErrorString(e));
  }
  // the posterior the last scoring round saw (mu never moves; sigma carries
  // the downdates of every pick before that round)
  hipError_t e = hipSuccess;
  if (mu_out) e = hipMemcpyAsync(mu_out, mu, (size_t)p * n * 4, hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess && sigma_out) e = hipMemcpyAsync(sigma_out, sd, (size_t)p * n * 4, hipMemcpyDeviceToDevice, s);
  if (e != hipSuccess) return fail(SCOOT_ERR_DEVICE, std::string("believer: ") + hipGetErrorString(e));
  return SCOOT_OK;
}

}  // namespace scoot
