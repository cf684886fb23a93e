// Internal declarations shared by the host code and the kernel launchers.
#pragma once

#include <algorithm>
#include <cmath>
#include <cstddef>
#include <cstdint>
#include <functional>
#include <string>
#include <vector>

#include "scoot.h"

namespace scoot {

// Granule the observation count is padded to (the posterior sizes its LDS
// and picks its wave count in units of it), the 16-row MFMA block of the
// triangular product, and the padded row stride of the scaled observations.
constexpr int kBlk32 = 32;
constexpr int kBlk16 = 16;
constexpr int kXsStride = 16;          // floats / doubles per observation row
constexpr double kPadCoord = 1.0e4;    // scaled coordinate of padding rows: k(x, pad) == 0

#ifdef __HIPCC__
#define SCOOT_HOST_DEVICE __host__ __device__
#else
#define SCOOT_HOST_DEVICE
#endif

// Waves per workgroup of the posterior: more than 9 granules of K*
// (72 KiB of LDS per 64-candidate tile) leave room for one workgroup per CU,
// so it gets 8 waves; otherwise two 4-wave workgroups share a CU.
inline int posterior_waves(int nb) { return nb > 9 ? 8 : 4; }

// Which 16-row blocks of V each wave of the posterior owns (both
// precisions).  Row block I costs I + 1 blocks of the triangle.  Plan entry p
// goes to wave p of a 4-wave workgroup; with 8 waves the two entries p and
// p + 4 share a SIMD and its matrix unit.  So the rows are first split into
// four sets of (nearly) equal cost, one per SIMD, by a depth-first search for
// the smallest capacity that admits a packing; with 8 waves each set is then
// halved between its two waves by an exact subset-sum split.  The packed
// inverse streams the blocks entry by entry, each entry's rows in increasing
// I, blocks J = 0..I.  Up to 36 row blocks: 6 bits per row in one 128-bit
// value held as two words (row k at bits 6k .. 6k + 5, lo the low word), so
// an entry holds up to 21 rows.
constexpr int kRowBits16 = 6;
constexpr int kMaxRows16 = 128 / kRowBits16;
struct RowPlan16 {
  uint64_t lo[8], hi[8];
  int32_t nrows[8];
  int32_t blk_start[9];
};

// Splits rows into two sets whose costs (I + 1) are as equal as possible.
inline void bisect_rows(const std::vector<int>& rows, std::vector<int>& lo, std::vector<int>& hi) {
  int total = 0;
  for (int I : rows) total += I + 1;
  // reach[k][s]: some subset of the first k rows costs s
  std::vector<std::vector<char>> reach(rows.size() + 1, std::vector<char>(total + 1, 0));
  reach[0][0] = 1;
  for (size_t k = 0; k < rows.size(); ++k)
    for (int s = 0; s <= total; ++s)
      if (reach[k][s]) {
        reach[k + 1][s] = 1;
        reach[k + 1][s + rows[k] + 1] = 1;
      }
  int best = 0;
  for (int s = 0; s <= total / 2; ++s)
    if (reach[rows.size()][s]) best = s;
  lo.clear();
  hi.clear();
  for (size_t k = rows.size(); k-- > 0;) {
    if (best >= rows[k] + 1 && reach[k][best - rows[k] - 1]) {
      lo.push_back(rows[k]);
      best -= rows[k] + 1;
    } else {
      hi.push_back(rows[k]);
    }
  }
}

// Places rows[k..] (decreasing) into four sets of cost at most cap.
inline bool pack_rows4(const std::vector<int>& rows, size_t k, int cap, int (&load)[4], std::vector<int> (&set)[4]) {
  if (k == rows.size()) return true;
  const int c = rows[k] + 1;
  for (int b = 0; b < 4; ++b) {
    bool same = false;  // a set with the same load was already tried
    for (int b2 = 0; b2 < b; ++b2) same = same || load[b2] == load[b];
    if (same || load[b] + c > cap) continue;
    load[b] += c;
    set[b].push_back(rows[k]);
    if (pack_rows4(rows, k + 1, cap, load, set)) return true;
    load[b] -= c;
    set[b].pop_back();
  }
  return false;
}

// The rows of each plan entry, each entry in increasing I.
inline void plan_entries(int nb, int W, std::vector<int> (&entry)[8]) {
  std::vector<int> all;
  for (int I = nb - 1; I >= 0; --I) all.push_back(I);
  std::vector<int> quarter[4];
  for (auto& e : entry) e.clear();
  for (int cap = (nb * (nb + 1) / 2 + 3) / 4;; ++cap) {
    int load[4] = {0, 0, 0, 0};
    for (auto& q : quarter) q.clear();
    if (pack_rows4(all, 0, cap, load, quarter)) break;
  }
  if (W == 8) {
    for (int q = 0; q < 4; ++q) bisect_rows(quarter[q], entry[q], entry[q + 4]);
  } else {
    for (int q = 0; q < 4; ++q) entry[q] = quarter[q];
  }
  for (auto& e : entry) std::sort(e.begin(), e.end());
}

// Entries of more than kMaxRows16 rows keep only their first kMaxRows16 (nrows
// tells; the launcher refuses such a plan).
inline RowPlan16 plan_rows16(int nb16, int W) {
  std::vector<int> entry[8];
  plan_entries(nb16, W, entry);
  RowPlan16 p{};
  int b = 0;
  for (int e = 0; e < 8; ++e) {
    const std::vector<int>& r = entry[e];
    p.blk_start[e] = b;
    p.nrows[e] = (int)r.size();
    unsigned __int128 v = 0;
    for (size_t k = 0; k < r.size(); ++k) {
      if ((int)k < kMaxRows16) v |= (unsigned __int128)r[k] << (kRowBits16 * k);
      b += r[k] + 1;
    }
    p.lo[e] = (uint64_t)v;
    p.hi[e] = (uint64_t)(v >> 64);
  }
  p.blk_start[8] = b;
  return p;
}
// Row q of entry e of a fp64 plan.
inline int plan16_row(const RowPlan16& p, int e, int q) {
  const unsigned __int128 v = ((unsigned __int128)p.hi[e] << 64) | p.lo[e];
  return (int)((v >> (kRowBits16 * q)) & ((1u << kRowBits16) - 1));
}

// Runs fn(c) for every chunk c = 0 .. n_chunks - 1 on the library's pool of
// host threads (the caller takes part) and returns when all have run.  The
// chunking is the caller's and must not depend on the thread count; fn must
// not call parallel_chunks itself.  Pool size: SCOOT_HOST_THREADS, else the
// hardware threads up to 16.
void parallel_chunks(int n_chunks, const std::function<void(int)>& fn);
// Threads of the pool, the caller included.
int pool_threads();
// While it lives, the parallel steps this thread starts take at most n pool
// workers besides itself (n < 0: no cap); results do not change.
class PoolHelpers {
 public:
  explicit PoolHelpers(int n);
  ~PoolHelpers();
  PoolHelpers(const PoolHelpers&) = delete;
  PoolHelpers& operator=(const PoolHelpers&) = delete;

 private:
  int prev_;
};

// In-place lower Cholesky factor of the m x m row-major A (the lower
// triangle is read; the upper is zeroed); false when a pivot is not positive
// or below 1e-13 of its diagonal entry.  Host threads, fixed chunking.
bool cholesky_lower(double* A, int m);
// L^-1 of a lower-triangular L (m x m row-major) into out (m x m, zero above
// the diagonal; transposed: out[j][i] = L^-1[i][j], zero below).
void lower_inverse(const double* L, int m, double* out, bool transposed);

void clear_error();
void set_error(const std::string& msg);
int fail(int status, const std::string& msg);
// As fail, for a message with static storage: allocates nothing.
int fail_static(int status, const char* msg);

// ---- fit (host) -----------------------------------------------------------
struct FitHost {
  int m = 0, d = 0, m_pad = 0, nb = 0;     // nb = m_pad / 32
  scoot_kernel kernel = SCOOT_MATERN52;
  double s2 = 1, tau2 = 0, c = 0;
  std::vector<double> L;                   // m x m row-major lower factor
  std::vector<double> Linv;                // m x m row-major lower inverse factor
  std::vector<double> alpha;               // m
  std::vector<double> scale;               // d: sqrt(2 nu) * log2(e) / l_k
  std::vector<double> Xw;                  // m x d observations after input warping (= X without)
  std::vector<double> warp_a, warp_b;      // d each, empty without warping
  double coef[3] = {0, 0, 0};              // k = (coef0 + u (coef1 + u coef2)) 2^-u
};

// Validates and computes K, its Cholesky factor, alpha and L^-1 in fp64.
// warp_a / warp_b: both null (no warping) or d positive values each.
int fit_host(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* ls,
             const double* warp_a, const double* warp_b, double s2, double tau2, double c, FitHost& out);
// fit_host's validation and everything but the factorization (L, Linv and
// alpha left empty).
int fit_setup(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* ls,
              const double* warp_a, const double* warp_b, double s2, double tau2, double c, FitHost& out);
// The device GP handle of a fit (its Linv and alpha filled): packing and upload.
int gp_from_fit(const FitHost& f, const double* warp_a, const double* warp_b, scoot_dtype dt, scoot_gp* out);
// mle_fit_device, then the GP at the optimum with L^-1 and alpha from the
// search's own device factorization (no host refit).
int mle_fit_device_gp(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                      const double* warp_b, double c, bool learn_warp, const double* lower, const double* upper,
                      int max_iter, double* theta, scoot_dtype dt, void* stream, scoot_gp* out);
// The GP at fixed hyperparameters with the factorization on the device.
int gp_fit_device(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* ls,
                  const double* warp_a, const double* warp_b, double s2, double tau2, double c, scoot_dtype dt,
                  void* stream, scoot_gp* out);

// Kumaraswamy input warping of one coordinate, w = 1 - (1 - x^a)^b, x clamped
// to [0, 1], without cancellation: ln x from log1p(x - 1) above 1/2,
// 1 - x^a = -expm1(a ln x), w = -expm1(b ln(1 - x^a)).
SCOOT_HOST_DEVICE inline double kumaraswamy(double x, double a, double b) {
  x = x < 0.0 ? 0.0 : (x > 1.0 ? 1.0 : x);
  const double lx = x > 0.5 ? log1p(x - 1.0) : log(x);
  return -expm1(b * log(-expm1(a * lx)));
}

// Maximum-likelihood hyperparameters (host_mle.cpp); theta = (log l_1..d, log s2, log tau2),
// followed by (log a_1..d, log b_1..d) when learn_warp (warp_a / warp_b must then be null).
int mle_nll(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
            const double* warp_b, double c, const double* theta, double* nll, double* grad,
            bool learn_warp = false);
int mle_fit(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
            const double* warp_b, double c, const double* lower, const double* upper, int max_iter, double* theta,
            double* nll, int* iterations, bool learn_warp = false);
// The inputs a likelihood evaluation sees, validated as mle_nll / mle_fit do:
// Xuse = the inputs warped by (warp_a, warp_b) when given, the raw inputs when
// the warp is learned; r = y - c.
int mle_inputs(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
               const double* warp_b, double c, bool learn_warp, std::vector<double>& Xuse, std::vector<double>& r);
// NLL and gradient at theta; false when K is not positive definite.
typedef std::function<bool(const double* theta, double* nll, double* grad)> NllFn;
// The box-constrained L-BFGS search of mle_fit over any evaluator of P parameters.
int lbfgs_box(const NllFn& nll_fn, int P, const double* lower, const double* upper, int max_iter, double* theta,
              double* nll_out, int* iters_out);
// mle_fit with every evaluation on the device (k_mle.hip), on `stream`.
int mle_fit_device(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                   const double* warp_b, double c, bool learn_warp, const double* lower, const double* upper,
                   int max_iter, double* theta, double* nll_out, int* iters_out, void* stream);
int mle_nll_device(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                   const double* warp_b, double c, bool learn_warp, const double* theta, double* nll, double* grad,
                   void* stream);

// Forest training (host_forest_train.cpp): tree-local child indices, preorder.
struct TrainedForest {
  std::vector<int32_t> feature, left, right;  // feature -1 at leaves
  std::vector<double> threshold, value;       // value: the node's weighted mean label
  std::vector<int64_t> tree_offset;           // n_trees + 1
};
int train_forest_host(const double* X, const double* y, int n, int d, int n_trees, int max_depth, uint64_t seed,
                      bool bootstrap, TrainedForest& out);

// Packs L^-1 into matrix-core A-operand order (see the posterior kernels).
void pack_linv_f32(const FitHost& f, std::vector<float>& out);
// The fp32 posterior's augmented observation rows (fp64 cross-term operand).
void pack_obs_f32(const FitHost& f, std::vector<double>& out);
void pack_linv_f64(const FitHost& f, std::vector<double>& out);

// ---- EHVI boxes (host) ------------------------------------------------------
struct BoxTable {
  int p = 0;
  int n_front = 0;
  std::vector<double> front;               // n_front x p, lexicographic
  std::vector<std::vector<double>> coord;  // per axis: [-inf, sorted unique front values..., ref]
  std::vector<int16_t> lo, hi;             // n_boxes x p coordinate indices (lo == 0 means -inf)
  int n_boxes() const { return p ? (int)lo.size() / p : 0; }
};
int build_boxes(const double* Y, int m, int p, const double* ref, BoxTable& out);

// ---- forest (host) ----------------------------------------------------------
// Packed node, 8 bytes: word0 = (child << 15) | (feature << 11), word1 = the
// threshold's float32 bits.  The two children of a node are adjacent (right =
// child + 1).  A leaf at position s stores child = s - 1 and, as threshold, a
// quiet NaN whose payload is the leaf's Q16 value: x <= NaN is false for every
// x, so a walk that reaches a leaf steps to s - 1 + 1 = s and stays there.
// Every chunk starts with one unused node, so no leaf sits at position 0.
// feature << 11 is the byte offset of that feature's column in the kernel's
// LDS copy of the candidates (512 threads x 4 bytes per feature).
constexpr int kForestThreadsPerBlock = 512;
constexpr uint32_t kLeafNaN = 0x7FC00000u;
constexpr int kChunkNodes = 8192;
struct ForestHost {
  int n_trees = 0, d = 0;
  std::vector<uint32_t> nodes;             // 2 words per node
  // Trees are packed in slots ordered by depth (deepest first, then by index),
  // so that the four trees a thread walks together have similar depths.
  std::vector<int32_t> tree_orig;          // tree index (as given) in each slot
  std::vector<uint32_t> root;              // packed index of each slot's root (n_trees + 1 entries)
  std::vector<uint32_t> depth;             // edges from each slot's root to its deepest leaf
  std::vector<int32_t> leaf_orig;          // per packed node: tree-local index of a leaf, -1 otherwise
  std::vector<int> chunk_tree;             // first slot of each LDS chunk (+ end)
  std::vector<uint32_t> chunk_first_node;  // packed index of each chunk's unused first node (+ end)
};
int pack_forest(const int32_t* feature, const float* threshold, const int32_t* left,
                const int32_t* right, const int32_t* leaf_q16, const int64_t* tree_offset,
                int n_trees, int d, ForestHost& out);

// ---- device state -----------------------------------------------------------
struct GPDevice {
  scoot_dtype dt = SCOOT_F32;
  int m = 0, d = 0, m_pad = 0, nb = 0;
  double s2 = 1, tau2 = 0, c = 0;
  void* buf = nullptr;        // one allocation holding everything below
  const void* linv = nullptr; // packed L^-1 (float or double)
  const void* xs = nullptr;   // fp32: the augmented observation rows (pack_obs_f32, double);
                              // fp64: m_pad x kXsStride scaled rows, alpha_i in column d when d < kXsStride
  const double* alpha = nullptr;  // m_pad
  const float* alpha32 = nullptr; // m_pad, float copy
  float scale32[SCOOT_MAX_DIM];
  double scale64[SCOOT_MAX_DIM];
  float coef32[3];
  double coef64[3];
  bool warp = false;              // candidates go through kumaraswamy(x, warp_a, warp_b) first
  double warp_a[SCOOT_MAX_DIM];
  double warp_b[SCOOT_MAX_DIM];
};

struct ForestDevice {
  int n_trees = 0, d = 0;
  uint32_t* nodes = nullptr;     // one allocation: nodes | root | depth | leaf_orig | tree_orig
  uint32_t* root = nullptr;
  uint32_t* depth = nullptr;
  int32_t* leaf_orig = nullptr;
  int32_t* tree_orig = nullptr;
  std::vector<int> chunk_tree;
  std::vector<uint32_t> chunk_first_node;
};

// Library-owned scratch of the current device, grown on demand.
void* device_scratch(size_t bytes, int slot);
// Lets `kernel` take up to the whole LDS of a CU (160 KiB) as dynamic LDS on
// the current device; done once per (device, kernel), thread-safe.
constexpr int kMaxLdsBytes = 160 * 1024;
int allow_full_lds(const void* kernel, const char* what);
// Pinned host staging for small uploads on a stream; the previous upload of
// the same slot is waited for before the buffer is reused.
int upload_async(void* dst, const void* src, size_t bytes, int slot, void* stream);

// ---- launchers (device) -----------------------------------------------------
// v_out (nullable, fp32 handles only): V = L^-1 K*^T, m_pad rows of n floats.
// With input warping (g.warp) the pool is warped first (fp32: into scratch by
// launch_warp_pool; fp64: inside the kernel), unless xc_warped says Xc already is.
int launch_posterior(const GPDevice& g, const float* Xc, int64_t n, void* mu, void* sigma,
                     const double* ei_c /* nullable: fused EI with c = best + xi */, void* ei,
                     void* stream, float* v_out = nullptr, bool xc_warped = false,
                     int64_t v_ld = 0 /* row stride of v_out; 0: n */);
int launch_warp_pool(const GPDevice& g, const float* Xc, int64_t n, float* out, void* stream);
int launch_ei(const void* mu, const void* sigma, int64_t n, scoot_dtype dt, double c, void* ei,
              void* stream);
int launch_ehvi(const void* const* mu, const void* const* sigma, int p, int64_t n, scoot_dtype dt,
                const BoxTable& boxes, void* ehvi, void* stream);
// EHVI followed by the masked top-q over it (mask nullable): for p <= 2 the
// first selection stage runs in the EHVI kernel's epilogue; as launch_ehvi
// then launch_topq otherwise.
int launch_ehvi_topq(const void* const* mu, const void* const* sigma, int p, int64_t n, scoot_dtype dt,
                     const BoxTable& boxes, void* ehvi, const uint8_t* mask, int q, int64_t* idx, void* score_out,
                     int32_t* n_valid, void* stream);
// mask[c] = votes >= vote_min and (known nullable) known[c] != 0.
int launch_forest(const ForestDevice& f, const float* Xc, int64_t n, int64_t vote_min,
                  int32_t* votes, uint8_t* mask, int32_t* leaf_idx, void* stream,
                  const uint8_t* known = nullptr);
// mask[i] = known ? (known[i] != 0) : 1.
int launch_mask_init(uint8_t* mask, const uint8_t* known, int64_t n, void* stream);
int launch_sobol_pool(const uint32_t* poly, const uint32_t* vinit, int d, const int32_t* levels, int64_t skip,
                      int64_t n, const double* A, const double* b, int r, float* Xc, uint8_t* known, void* stream);
int launch_known_constraints(const float* Xc, int64_t n, int d, const double* A, const double* b, int r,
                             uint8_t* known, void* stream);
int launch_topq(const void* score, const uint8_t* mask, int64_t n, scoot_dtype dt, int q,
                int64_t* idx, void* score_out, int32_t* n_valid, void* stream);
// As launch_topq, with the stage-1 lists in a fixed device array: allocates nothing.
int launch_topq_static(const void* score, const uint8_t* mask, int64_t n, scoot_dtype dt, int q, int64_t* idx,
                       void* score_out, int32_t* n_valid, void* stream);
// Stage 2 of top-q alone, over n_parts lists of q keys (Key64 for F32,
// Key128 for F64) and their eligible counts, written by a fused producer.
int launch_topq_stage2(const void* score, scoot_dtype dt, int n_parts, int q, const void* part_keys,
                       const int32_t* part_count, int64_t* idx, void* score_out, int32_t* n_valid, void* stream);
int launch_random_pick(const uint8_t* flags, int64_t n, uint64_t seed, int q, int64_t* idx, int32_t* n_flagged,
                       void* stream);
int launch_mace_scores(const void* mu, const void* sigma, int64_t n, scoot_dtype dt, double c, double beta, void* ucb,
                       void* pi, void* ei, void* stream);
int launch_pareto_front3(const void* a, const void* b, const void* c, const uint8_t* mask, int64_t n, scoot_dtype dt,
                         uint8_t* front, int32_t* n_front, void* stream);

// Sequential Kriging-believer picks (fp32 GPs only).
size_t kb_workspace_bytes(const GPDevice* const* g, int p, int64_t n, int q);
int run_kriging_believer(const GPDevice* const* g, int p, const ForestDevice* f, const uint8_t* known,
                         int64_t vote_min, const float* Xc, int64_t n, const double* Y_obs, int m_obs, const double* ref, int q, void* ws,
                         int64_t* picks, double* pick_acq, int* n_picked, float* mu_out, float* sigma_out,
                         void* stream);

}  // namespace scoot
