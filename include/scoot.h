/*
 * scoot.h -- C ABI of the MI355X (gfx950) candidate-scoring library.
 *
 * The library scores a pool of candidate engine configurations the way the
 * suggestion step of SCOOT (SLO-Oriented Performance Tuning for LLM Inference
 * Engines) does: GP posterior per objective (Sec. 4.3, Eq. 4-5), acquisition
 * (EI, Eq. 8; EHVI, Eq. 9), the random-forest hidden-constraint mask
 * POF(x) >= Delta (Eq. 3, Sec. 4.7) and the top-q parallel pick (Sec. 4.6).
 * Observed configurations and SLO values go in; indices of the next
 * configurations to evaluate come out.
 *
 * Conventions shared by every call
 * --------------------------------
 * - Every objective is MINIMISED.  The paper maximises lambda * f (Eq. 1); pass
 *   y = -lambda * f.  The EHVI reference point is therefore an upper bound.
 * - Arrays of candidate length n (pool, mu, sigma, scores, votes, mask, leaf
 *   ids) and the q-sized outputs are DEVICE pointers owned by the caller.
 *   Everything else (observations, hyperparameters, forest arrays, reference
 *   point) is a HOST pointer, read during the call and not retained.
 * - The candidate pool Xc is n x d float32, row-major, on the device.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Device
 *   work is enqueued asynchronously on it; the caller synchronises.  Calls
 *   that use one device must be issued on one stream, or the caller orders
 *   them: library-owned scratch of a device is reused from call to call.
 * - Handles are library-owned and not thread-safe; destroy them with the
 *   matching *_destroy call.
 * - Host-side steps (GP fit, likelihood and its search, forest training) run
 *   on a pool of host threads the library starts on first use
 *   (SCOOT_HOST_THREADS, else the hardware threads up to 16).  Their results
 *   do not depend on the thread count, and calls that share no handle may run
 *   from several threads at once (scoot_suggest runs its objectives' searches
 *   that way).
 * - Every call returns a scoot_status.  On error the outputs are undefined and
 *   scoot_last_error() returns a message for the calling thread.  No C++
 *   exception crosses the ABI.
 */
#ifndef SCOOT_H
#define SCOOT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SCOOT_ABI_VERSION 5

typedef enum scoot_dtype { SCOOT_F32 = 0, SCOOT_F64 = 1 } scoot_dtype;

/* Covariance of a GP (scoot_gp_fit_ex). */
typedef enum scoot_kernel { SCOOT_MATERN52 = 0, SCOOT_MATERN32 = 1 } scoot_kernel;

typedef enum scoot_status {
  SCOOT_OK = 0,
  SCOOT_ERR_INVALID_ARG = -1, /* bad shape, null pointer, NaN/Inf host input, q out of range */
  SCOOT_ERR_NOT_PD = -2,      /* K + tau^2 I is not numerically positive definite */
  SCOOT_ERR_DEVICE = -3,      /* a HIP runtime call failed; see scoot_last_error() */
  SCOOT_ERR_UNSUPPORTED = -4, /* size beyond the limits stated below */
  SCOOT_ERR_NO_MEMORY = -5    /* host or device allocation failed */
} scoot_status;

/* Limits of this build. */
#define SCOOT_MAX_DIM 16        /* d: parameters per configuration */
#define SCOOT_MAX_OBS 576       /* m: observations per GP */
#define SCOOT_MAX_OBJECTIVES 3  /* p */
#define SCOOT_MAX_Q 64          /* q: picks per suggestion */
#define SCOOT_MAX_TREES 32767   /* T: trees per forest (votes fit int32) */
#define SCOOT_MAX_CONSTRAINTS 8 /* r: known-constraint rows */
#define SCOOT_SOBOL_MAX_DEGREE 18 /* degree of a Sobol dimension's polynomial; vinit row stride */

typedef struct scoot_gp_t* scoot_gp;
typedef struct scoot_forest_t* scoot_forest;

/* Version of this header's ABI (SCOOT_ABI_VERSION). */
int scoot_abi_version(void);

/* Static text for a status code. */
const char* scoot_status_string(int status);

/* Message describing the last failing call made by this thread ("" if none). */
const char* scoot_last_error(void);

/* ---------------------------------------------------------------------------
 * Fit (host).  Sec. 4.3, Eq. 4-5: K = k(X, X) + tau^2 I with the Matern-5/2
 * ARD covariance k(x, x') = s2 (1 + sqrt5 r + 5 r^2 / 3) exp(-sqrt5 r),
 * r^2 = sum_k ((x_k - x'_k) / l_k)^2; L = chol(K); alpha = K^-1 (y - c).
 * The _ex calls also take the paper's own covariance (Sec. 4.3): kernel =
 * SCOOT_MATERN32, k = s2 (1 + sqrt3 r) exp(-sqrt3 r), and input warping:
 * warp_a, warp_b [d] > 0 (both or neither; NULL = none) put every input
 * dimension through the Kumaraswamy distribution function
 * w(x) = 1 - (1 - x^a)^b, x clamped to [0, 1], before the covariance -- for
 * the observations here and for every candidate in scoot_posterior (and the
 * calls built on it); the forest mask still sees the raw candidates.
 *
 * scoot_gp_factor_host: host-only arithmetic of the fit, for inspection.
 *   X      [m*d] observed configurations, row-major, finite.
 *   y      [m]   observed values of one objective, finite.
 *   lengthscale [d] > 0; signal_var s2 > 0; noise_var tau^2 >= 0;
 *   prior_mean c (Eq. 4 has c = 0).
 *   L      [m*m] out: lower Cholesky factor, row-major (upper part zeroed).
 *   alpha  [m]   out.
 *   Errors: INVALID_ARG, UNSUPPORTED (m > SCOOT_MAX_OBS, d > SCOOT_MAX_DIM),
 *   NOT_PD.
 *
 * scoot_gp_fit: the same fit, then a device-resident GP state (the inverse
 *   factor L^-1 packed for the matrix cores, scaled observations, alpha) on the
 *   current HIP device, uploaded synchronously (`stream` is not used).  dt
 *   selects the precision of scoot_posterior for this handle.  *out receives
 *   the handle.
 * ------------------------------------------------------------------------- */
int scoot_gp_factor_host(const double* X, const double* y, int m, int d, const double* lengthscale,
                         double signal_var, double noise_var, double prior_mean, double* L,
                         double* alpha);
int scoot_gp_fit(const double* X, const double* y, int m, int d, const double* lengthscale,
                 double signal_var, double noise_var, double prior_mean, scoot_dtype dt,
                 void* stream, scoot_gp* out);
int scoot_gp_factor_host_ex(const double* X, const double* y, int m, int d, scoot_kernel kernel,
                            const double* lengthscale, const double* warp_a, const double* warp_b,
                            double signal_var, double noise_var, double prior_mean, double* L, double* alpha);
int scoot_gp_fit_ex(const double* X, const double* y, int m, int d, scoot_kernel kernel,
                    const double* lengthscale, const double* warp_a, const double* warp_b, double signal_var,
                    double noise_var, double prior_mean, scoot_dtype dt, void* stream, scoot_gp* out);
/* scoot_gp_fit_device: scoot_gp_fit_ex with K, its Cholesky factor, L^-1 and
 * alpha computed on the current device (fp64, the kernels of
 * scoot_gp_nll_device, on `stream`), then packed and uploaded as there; the
 * state agrees with scoot_gp_fit_ex's to rounding.  noise_var must be > 0.
 * Errors: as scoot_gp_fit_ex; INVALID_ARG also for noise_var <= 0; DEVICE for
 * a failed allocation or launch. */
int scoot_gp_fit_device(const double* X, const double* y, int m, int d, scoot_kernel kernel,
                        const double* lengthscale, const double* warp_a, const double* warp_b, double signal_var,
                        double noise_var, double prior_mean, scoot_dtype dt, void* stream, scoot_gp* out);
int scoot_gp_destroy(scoot_gp gp);

/* ---------------------------------------------------------------------------
 * Maximum-likelihood hyperparameters (host, fp64).  Sec. 4.3: SCOOT learns the
 * noise level tau^2 by maximum likelihood; the lengthscales and the signal
 * variance are learned with it.  theta [d + 2] = (log l_1 .. log l_d,
 * log s2, log tau2); X, y, kernel, warp_a/warp_b and prior_mean as in
 * scoot_gp_fit_ex.
 *
 * scoot_gp_nll: nll = 1/2 r^T K^-1 r + 1/2 log det K + m/2 log(2 pi) with
 *   r = y - prior_mean, K = k_theta(X, X) + tau^2 I, and grad [d + 2]
 *   (nullable) its gradient in theta.
 * scoot_gp_mle: minimises nll over the box lower <= theta <= upper ([d + 2]
 *   each; lower == upper holds a parameter fixed) from the theta given
 *   (in/out): L-BFGS over theta = lower + (upper - lower) sigmoid(z), so every
 *   iterate stays inside the box; stops when the gradient in z is below 1e-9,
 *   the decrease per iteration is below 1e-13 of |nll|, no step decreases
 *   nll, or after max_iter iterations.  nll (nullable) receives the final
 *   value, iterations (nullable) the count.  Work per evaluation: a Cholesky
 *   factorisation and an inverse of the m x m K (about m^3 flops).
 * Errors: INVALID_ARG, UNSUPPORTED, NOT_PD (K not positive definite at the
 *   start), NO_MEMORY.
 * ------------------------------------------------------------------------- */
int scoot_gp_nll(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                 const double* warp_b, double prior_mean, const double* theta, double* nll, double* grad);
int scoot_gp_mle(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                 const double* warp_b, double prior_mean, const double* lower, const double* upper, int max_iter,
                 double* theta, double* nll, int* iterations);

/* ---------------------------------------------------------------------------
 * As scoot_gp_nll and scoot_gp_mle with the input warping learned as well
 * (Sec. 4.3: the paper's covariance is Matern-3/2 with input warping after
 * Snoek et al., whose warp parameters are fitted together with the GP).
 * theta [3d + 2] = (log l_1..d, log s2, log tau2, log a_1..d, log b_1..d):
 * every input x passes through w = 1 - (1 - x^a_k)^b_k (x clamped to [0, 1])
 * before the covariance sees it, and grad [3d + 2] (nullable) is the
 * analytic gradient in all of them (through the warped inputs:
 * dK_ij/dlog a_k = -R_ij (w_ik - w_jk)(dw_ik - dw_jk)/l_k^2 with R the radial
 * factor of the lengthscale derivatives).  lower, upper [3d + 2] as in
 * scoot_gp_mle.  The learned (a, b) go to scoot_gp_fit_ex as warp_a, warp_b.
 * Errors: as scoot_gp_nll / scoot_gp_mle.
 * ------------------------------------------------------------------------- */
int scoot_gp_nll_warp(const double* X, const double* y, int m, int d, scoot_kernel kernel, double prior_mean,
                      const double* theta, double* nll, double* grad);
int scoot_gp_mle_warp(const double* X, const double* y, int m, int d, scoot_kernel kernel, double prior_mean,
                      const double* lower, const double* upper, int max_iter, double* theta, double* nll,
                      int* iterations);

/* ---------------------------------------------------------------------------
 * The likelihood of Sec. 4.3 evaluated on the current device (fp64), and the
 * search with every evaluation there.  Arguments as scoot_gp_nll /
 * scoot_gp_mle (host pointers in and out; the library uploads X and y once
 * and reads back the value and gradient per evaluation); learn_warp = 0:
 * theta [d + 2] with the fixed warp_a/warp_b (nullable); learn_warp = 1:
 * theta, lower, upper [3d + 2] as in scoot_gp_nll_warp, warp_a and warp_b
 * must be NULL.  The work of an evaluation runs on `stream` (NULL: the null
 * stream) and the call returns after it: K, its Cholesky factor by 16 x 16
 * blocks (products on the fp64 matrix cores) with u = L^-1 r alongside, the NLL
 * from the pivots and u; with grad (nullable) also L^-1, alpha = L^-T u, K^-1
 * and the gradient's trace terms.  Results agree with the
 * host calls to rounding (same definitions, other summation order).  The
 * search is the host's L-BFGS (same stopping rules) and allocates its device
 * work space (about 16 m^2 bytes) once per call.
 * Errors: as scoot_gp_nll / scoot_gp_mle; INVALID_ARG also for learn_warp
 *   with a fixed warp given; DEVICE for a failed allocation or launch.
 * ------------------------------------------------------------------------- */
int scoot_gp_nll_device(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                        const double* warp_b, double prior_mean, int learn_warp, const double* theta, double* nll,
                        double* grad, void* stream);
int scoot_gp_mle_device(const double* X, const double* y, int m, int d, scoot_kernel kernel, const double* warp_a,
                        const double* warp_b, double prior_mean, int learn_warp, const double* lower,
                        const double* upper, int max_iter, double* theta, double* nll, int* iterations,
                        void* stream);

/* ---------------------------------------------------------------------------
 * Posterior (device).  Eq. 4 and Eq. 5 of Sec. 4.3 at every candidate:
 *   mu[i]    = c + k(x_i, X) alpha
 *   sigma[i] = sqrt(max(0, s2 - ||L^-1 k(X, x_i)||^2))   (latent f; tau^2 not added)
 * Xc [n*d] float32 device (d = the fitted d); mu, sigma [n] device, float32 or
 * float64 per the handle's dtype.  n = 0 is a no-op.  A NaN in a candidate row
 * gives NaN mu/sigma for that candidate.
 * Errors: INVALID_ARG (null handle/pointer, n < 0), DEVICE.
 * ------------------------------------------------------------------------- */
int scoot_posterior(scoot_gp gp, const float* Xc, int64_t n, void* mu, void* sigma, void* stream);

/* ---------------------------------------------------------------------------
 * Expected improvement (device), Eq. 8 of Sec. 4.4.1 mirrored to minimisation:
 *   ei[i] = E[max(0, best_y + xi - Y_i)],  Y_i ~ N(mu[i], sigma[i]^2)
 *         = (c - mu) Phi(u) + sigma phi(u),  c = best_y + xi, u = (c - mu) / sigma,
 * and max(0, c - mu) where sigma = 0.  The paper fixes xi = 1e-4 (Sec. 4.5.1).
 * mu, sigma, ei [n] device of type dt.  Errors: INVALID_ARG, DEVICE.
 * ------------------------------------------------------------------------- */
int scoot_acq_ei(const void* mu, const void* sigma, int64_t n, scoot_dtype dt, double best_y, double xi,
                 void* ei, void* stream);

/* ---------------------------------------------------------------------------
 * Expected hypervolume improvement, Eq. 9 of Sec. 4.4.2 (HV of Fig. 4).
 *
 * scoot_ehvi_front (host): the front of Y_obs [m_obs*p] (row-major) w.r.t. ref
 *   [p]: rows strictly below ref in every objective that no other row weakly
 *   dominates, duplicates once, sorted lexicographically into front
 *   [m_obs*p] (nullable); *n_front receives its size and *n_boxes (nullable)
 *   the number of boxes the device kernel sums over.
 *
 * scoot_acq_ehvi (device): for every candidate,
 *   ehvi[i] = E[HV(P + {Y_i}) - HV(P)] = sum_B prod_j (G_j(u_Bj) - G_j(l_Bj)),
 *   G_j(c) = E[(c - Y_ij)^+], over boxes B = [l, u] partitioning the region
 *   below ref that the front P leaves open (G(-inf) = 0).
 *   mu, sigma: arrays of p device pointers, each [n] of type dt.  p in 1..3.
 *   Y_obs, ref: host.  ehvi [n] device.
 * Errors: INVALID_ARG, UNSUPPORTED (front too large for the on-chip tables),
 * DEVICE.
 * ------------------------------------------------------------------------- */
int scoot_ehvi_front(const double* Y_obs, int m_obs, int p, const double* ref, double* front,
                     int* n_front, int* n_boxes);
int scoot_acq_ehvi(const void* const* mu, const void* const* sigma, int p, int64_t n, scoot_dtype dt,
                   const double* Y_obs, int m_obs, const double* ref, void* ehvi, void* stream);

/* ---------------------------------------------------------------------------
 * Random-forest probability of feasibility (Sec. 4.7) and the mask of Eq. 3.
 *
 * scoot_forest_create: n_trees regression trees as flat host arrays; tree t
 *   owns nodes tree_offset[t] .. tree_offset[t+1]-1 (tree_offset has
 *   n_trees+1 entries, tree_offset[0] = 0).  left/right are tree-local child
 *   indices, -1 at a leaf (both or neither).  feature in [0, d) at internal
 *   nodes; threshold float32; leaf_q16 = round(leaf value * 65536) at leaves,
 *   in [0, 65536].  Every tree must be a tree rooted at its first node.  The
 *   forest is validated, repacked (children adjacent) and uploaded
 *   synchronously to the current device.
 *
 * scoot_vote_threshold (host): the smallest vote count with POF >= delta,
 *   ceil(delta * (n_trees * 65536)) computed in double precision.
 *
 * scoot_rf_feasibility (device): each tree is walked from its root, left iff
 *   x[feature] <= threshold (float32 compare; NaN goes right), to a leaf;
 *   votes[i] = sum of the reached leaves' Q16 values (exact int32);
 *   mask[i] = votes[i] >= scoot_vote_threshold(delta, T);
 *   leaf_idx [n*n_trees] (nullable) = tree-local index of the reached leaf.
 *   Xc [n*d] float32 device; votes [n] int32 device (nullable); mask [n] u8
 *   device (nullable).  delta in [0, 1].
 * Errors: INVALID_ARG, UNSUPPORTED, DEVICE, NO_MEMORY.
 * ------------------------------------------------------------------------- */
int scoot_forest_create(const int32_t* feature, const float* threshold, const int32_t* left,
                        const int32_t* right, const int32_t* leaf_q16, const int64_t* tree_offset,
                        int n_trees, int d, scoot_forest* out);
int scoot_forest_destroy(scoot_forest f);

/* ---------------------------------------------------------------------------
 * Training the feasibility forest (host; Sec. 4.7: a random forest regressor
 * on every evaluated configuration, y = 1 ran, 0 crashed).  X [n*d] row-major,
 * y [n], finite.  Each of the n_trees trees is grown by exhaustive search on
 * the float32-rounded features: a node splits on the feature and threshold
 * maximising sum_L^2 / w_L + sum_R^2 / w_R (weighted label sums and weights),
 * threshold a/2 + b/2 between consecutive distinct values a < b (a if that
 * rounds up to b); equal scores go to the lower feature, then the lower
 * threshold; a node is a leaf (value: weighted mean label) at max_depth
 * (0 .. 64), with fewer than two distinct samples, when its labels are all
 * equal, or when no split beats the unsplit node.  bootstrap != 0: tree t
 * trains on draws floor(u n), u = (output t n + j of SplitMix64 from seed,
 * j = 0 .. n-1) >> 11 over 2^53, each with its multiplicity; otherwise on
 * every draw once.  All features are considered at every split.
 *
 * scoot_forest_train: the trees as flat arrays, nodes in preorder (left child
 *   first), child indices tree-local, -1 at leaves: feature (-1 at leaves),
 *   threshold (double), left, right, value (double) [capacity];
 *   tree_offset [n_trees + 1]; *n_nodes = the node count.  feature == NULL:
 *   only the count is reported.
 * scoot_forest_train_create: trains, then scoot_forest_create on the device
 *   format (thresholds rounded down to float32, leaves round(value * 65536)
 *   half to even).
 * Errors: INVALID_ARG (null, non-finite input, bad sizes, capacity below the
 *   count), UNSUPPORTED (d > SCOOT_MAX_DIM, a tree above 8191 nodes), and
 *   those of scoot_forest_create.
 * ------------------------------------------------------------------------- */
int scoot_forest_train(const double* X, const double* y, int n, int d, int n_trees, int max_depth, uint64_t seed,
                       int bootstrap, int64_t capacity, int32_t* feature, double* threshold, int32_t* left,
                       int32_t* right, double* value, int64_t* tree_offset, int64_t* n_nodes);
int scoot_forest_train_create(const double* X, const double* y, int n, int d, int n_trees, int max_depth,
                              uint64_t seed, int bootstrap, scoot_forest* out);
int scoot_vote_threshold(double delta, int n_trees, int64_t* votes_min);
int scoot_rf_feasibility(scoot_forest f, const float* Xc, int64_t n, double delta, int32_t* votes,
                         uint8_t* mask, int32_t* leaf_idx, void* stream);

/* ---------------------------------------------------------------------------
 * Top-q parallel suggestion (Sec. 4.6): the q eligible candidates with the
 * largest score, score descending, lowest index first on ties (-0 == +0).
 * Eligible = mask[i] != 0 (mask nullable: all) and score[i] is not NaN.
 * score [n] device of type dt; idx [q] int64 device; score_out [q] device of
 * type dt (nullable); n_valid [1] int32 device (nullable) = number eligible.
 * Fewer than q eligible: the tail of idx is -1 and of score_out NaN (the paper
 * fills that shortfall with Sobol points, a step left to the caller).
 * 1 <= q <= SCOOT_MAX_Q; 0 <= n < 2^31.
 * Errors: INVALID_ARG, DEVICE, NO_MEMORY.
 * ------------------------------------------------------------------------- */
int scoot_suggest_topq(const void* score, const uint8_t* mask, int64_t n, scoot_dtype dt, int q,
                       int64_t* idx, void* score_out, int32_t* n_valid, void* stream);

/* ---------------------------------------------------------------------------
 * scoot_suggest_topq for callers that cannot allocate memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same arguments, kernels and results, but the selection's intermediate lists
 * live in one fixed device array of 327,680 bytes per GPU (enough for every
 * n < 2^31 and q <= SCOOT_MAX_Q), held from the first call on that GPU until
 * the process ends, instead of the library's grow-only scratch.  The call
 * allocates no host or device memory, also on its error paths.  Every call on
 * one GPU uses that GPU's array: calls that overlap on one GPU (other streams,
 * other host threads) race and must be serialised by the caller.  Each call
 * writes every entry it later reads, so no clearing between calls is needed.
 * Errors: INVALID_ARG (as scoot_suggest_topq), UNSUPPORTED (lists larger than
 * the array; cannot happen within the limits above), DEVICE.
 * ------------------------------------------------------------------------- */
int scoot_suggest_topq_noalloc(const void* score, const uint8_t* mask, int64_t n, scoot_dtype dt, int q,
                               int64_t* idx, void* score_out, int32_t* n_valid, void* stream);

/* ---------------------------------------------------------------------------
 * Adaptation of Delta after a batch of k evaluated suggestions (Algorithm 1,
 * Sec. 4.7), host only.  Some result invalid: Delta = min(0.75, max(0.5,
 * Delta + 0.05)), c = 0.  Otherwise c += k and, if c >= 5, Delta =
 * max(0.25, Delta - 0.05), c -= 5.  Errors: INVALID_ARG (null, k < 0).
 * ------------------------------------------------------------------------- */
int scoot_delta_update(double* delta, int* c, int k, int any_invalid);

/* ---------------------------------------------------------------------------
 * One whole scoring pass (Sec. 4.1 steps 3-8): scoot_posterior for each of
 * the p GPs, EI (p = 1, with best_y and xi) or EHVI (p >= 2, with Y_obs
 * [m_obs*p] and ref [p]), scoot_rf_feasibility with delta (f nullable: every
 * candidate feasible) and scoot_suggest_topq on the acquisition.
 * mu, sigma: [p*n] device (objective-major) of the GPs' dtype (all equal);
 * acq [n]; votes [n] (nullable); mask [n]; idx [q]; score_out [q] (nullable);
 * n_valid [1] (nullable).  Errors: as the calls it makes.
 * ------------------------------------------------------------------------- */
int scoot_score_pool(const scoot_gp* gps, int p, scoot_forest f, const float* Xc, int64_t n,
                     double best_y, double xi, const double* Y_obs, int m_obs, const double* ref,
                     double delta, int q, void* mu, void* sigma, void* acq, int32_t* votes,
                     uint8_t* mask, int64_t* idx, void* score_out, int32_t* n_valid, void* stream);
/* As scoot_score_pool, with the known-constraint mask of the pool (known [n]
 * u8 device, nullable = every candidate admissible, e.g. from scoot_sobol_pool
 * or scoot_known_constraints) folded into the mask: mask[i] = feasible and
 * known[i] != 0. */
int scoot_score_pool_ex(const scoot_gp* gps, int p, scoot_forest f, const uint8_t* known, const float* Xc,
                        int64_t n, double best_y, double xi, const double* Y_obs, int m_obs, const double* ref,
                        double delta, int q, void* mu, void* sigma, void* acq, int32_t* votes, uint8_t* mask,
                        int64_t* idx, void* score_out, int32_t* n_valid, void* stream);

/* ---------------------------------------------------------------------------
 * Sequential Kriging-believer suggestion of q candidates, an extension of the
 * parallel suggestion of Sec. 4.6 (the paper takes the top k at once).  Each
 * pick maximises EHVI (Eq. 9, p = 1..3) over the feasible (Eq. 3 with delta;
 * f nullable: all feasible), not yet picked candidates; the pick then joins
 * the observations with its posterior mean as a fantasy value and noise
 * tau^2: the Cholesky factor is extended by one row, V = L^-1 K*^T gains the
 * row (k(x, x_p) - v_p^T V[:, x]) / d, sigma^2 drops by its square, the mean
 * stays, and the front gains the fantasy.  Ties go to the lowest index.
 *
 * gps: p fp32 handles (fp64: UNSUPPORTED) sharing d.  Xc [n*d] device.
 * Y_obs [m_obs*p], ref [p]: host.  workspace: device, at least the size
 * scoot_suggest_kb_workspace returns (it holds V of every objective: about
 * 4 (m + q) n p bytes); NULL: the library allocates and frees it in the call.
 * picks [q], pick_acq [q] (nullable), n_picked: HOST outputs — the call
 * synchronises `stream` after every pick.  Fewer than q feasible candidates:
 * *n_picked < q and the tail of picks is untouched.
 * Errors: INVALID_ARG, UNSUPPORTED, NO_MEMORY, DEVICE.
 * ------------------------------------------------------------------------- */
int scoot_suggest_kb_workspace(const scoot_gp* gps, int p, int64_t n, int q, uint64_t* bytes);
int scoot_suggest_kb(const scoot_gp* gps, int p, scoot_forest f, const float* Xc, int64_t n,
                     const double* Y_obs, int m_obs, const double* ref, double delta, int q, void* workspace,
                     uint64_t workspace_bytes, int64_t* picks, double* pick_acq, int* n_picked, void* stream);
/* As scoot_suggest_kb; known [n] u8 device (nullable) restricts the
 * eligible candidates to the admissible ones, as in scoot_score_pool_ex.
 * mu_out, sigma_out [p*n] float32 device (objective-major, each nullable):
 * the posterior the last scoring round was computed from — the mean of the
 * observations (unchanged by the fantasies) and the standard deviation after
 * the fantasies of every pick before that round (q - 1 of them when all q
 * picks are made, *n_picked of them on a shortfall). */
int scoot_suggest_kb_ex(const scoot_gp* gps, int p, scoot_forest f, const uint8_t* known, const float* Xc,
                        int64_t n, const double* Y_obs, int m_obs, const double* ref, double delta, int q,
                        void* workspace, uint64_t workspace_bytes, int64_t* picks, double* pick_acq, int* n_picked,
                        float* mu_out, float* sigma_out, void* stream);

/* ---------------------------------------------------------------------------
 * MACE suggestion for one objective (Sec. 4.5.1: UCB, PI and EI, their Pareto
 * front over the candidates, k of them drawn at random; Sec. 4.6).  The
 * objective is minimised, so with best = best_y + xi and Y ~ N(mu, sigma^2):
 *
 * scoot_ucb_beta (host): the paper's schedule beta_t = 2 log(t^2 pi^2 /
 *   (6 delta)), delta = 1 / t^2, for tuning iteration t >= 1.  The paper
 *   multiplies sigma by this beta itself (Eq. 6); GP-UCB proper uses its square
 *   root -- the scoring calls take the multiplier as given.
 *
 * scoot_acq_mace (device): ucb = beta * sigma - mu (Eq. 6 for -Y), pi =
 *   P(Y < best) (Eq. 7; 1 or 0 when sigma = 0), ei = E[(best - Y)^+] (Eq. 8).
 *   mu, sigma, ucb, pi, ei: [n] device arrays of type dt.
 *
 * scoot_pareto_front3 (device): front[i] = 1 when candidate i is eligible
 *   (mask[i] != 0, mask nullable = all; no NaN score) and no eligible
 *   candidate scores at least as high on all of a, b, c and higher on one (all
 *   maximised; equal score vectors do not dominate each other), else 0.
 *   a, b, c [n] device of type dt; front [n] u8 device; n_front [1] int32
 *   device (nullable) = number of front members.  0 <= n < 2^31.  Worst-case
 *   work grows with the square of the number of candidates that survive a
 *   1024-candidate tile.
 *
 * scoot_random_pick (device): the q flagged candidates (flags[i] != 0) with
 *   the largest u_i, u_i = output number i (0-based) of SplitMix64 started
 *   from seed (state advanced by 0x9E3779B97F4A7C15, Stafford's finaliser);
 *   lower index first on equal draws.  That is a uniformly random q-subset of
 *   the flagged set, in random order, reproducible from (seed, flags).
 *   idx [q] int64 device (tail -1 when fewer are flagged); n_flagged [1] int32
 *   device (nullable).  1 <= q <= SCOOT_MAX_Q; 0 <= n < 2^31.
 *
 * scoot_suggest_mace (device): scoot_posterior, scoot_acq_mace,
 *   scoot_rf_feasibility with delta (f nullable: all feasible),
 *   scoot_pareto_front3 on (ucb, pi, ei) under the mask, scoot_random_pick
 *   of q from the front.  mu, sigma, ucb, pi, ei [n] of the GP's dtype; votes
 *   [n] (nullable); mask, front [n] u8; idx [q]; n_front [1] (nullable).
 *
 * Errors: INVALID_ARG (null pointer, bad dtype, n or q out of range, non-finite
 * best_y, xi or beta, t < 1), DEVICE, NO_MEMORY, and those of the calls made.
 * ------------------------------------------------------------------------- */
int scoot_ucb_beta(int t, double* beta);
int scoot_acq_mace(const void* mu, const void* sigma, int64_t n, scoot_dtype dt, double best_y, double xi,
                   double beta, void* ucb, void* pi, void* ei, void* stream);
int scoot_pareto_front3(const void* a, const void* b, const void* c, const uint8_t* mask, int64_t n,
                        scoot_dtype dt, uint8_t* front, int32_t* n_front, void* stream);
int scoot_random_pick(const uint8_t* flags, int64_t n, uint64_t seed, int q, int64_t* idx, int32_t* n_flagged,
                      void* stream);
int scoot_suggest_mace(scoot_gp gp, scoot_forest f, const float* Xc, int64_t n, double best_y, double xi,
                       double beta, double delta, uint64_t seed, int q, void* mu, void* sigma, void* ucb,
                       void* pi, void* ei, int32_t* votes, uint8_t* mask, uint8_t* front, int64_t* idx,
                       int32_t* n_front, void* stream);
/* As scoot_suggest_mace; known [n] u8 device (nullable) is ANDed into the
 * mask, as in scoot_score_pool_ex. */
int scoot_suggest_mace_ex(scoot_gp gp, scoot_forest f, const uint8_t* known, const float* Xc, int64_t n,
                          double best_y, double xi, double beta, double delta, uint64_t seed, int q, void* mu,
                          void* sigma, void* ucb, void* pi, void* ei, int32_t* votes, uint8_t* mask,
                          uint8_t* front, int64_t* idx, int32_t* n_front, void* stream);

/* ---------------------------------------------------------------------------
 * Candidate generation and known constraints (Sec. 4.5.3: the optimiser's
 * space is pruned by constraints known in advance, listed per engine in the
 * appendix; Sec. 4.7: a shortfall of suggestions is filled with Sobol points;
 * Sec. 4.1 and Algorithm 1: the first observations are Sobol points).
 *
 * scoot_sobol_pool (device): rows i = 0..n-1 of Xc [n*d] float32 are Sobol
 *   points skip + i (Bratley-Fox direction numbers, Gray-code order, 32-bit:
 *   coordinate j of point t is the XOR of V_j[k] over the set bits k of
 *   t ^ (t >> 1), over 2^32) rounded to the space's grids: levels[j] = 0
 *   continuous, 1 boolean (1 when the coordinate is >= 1/2), L >= 2 the grid
 *   k / (L - 1) (rint in double, half to even), then stored as float32.
 *   Dimension j is given by poly[j], the primitive polynomial over GF(2) as
 *   the integer whose bit t is the coefficient of x^t (1 = degree 0, the van
 *   der Corput sequence), and its initial direction numbers m_1..m_s (s the
 *   degree) in vinit[j * SCOOT_SOBOL_MAX_DEGREE + 0 .. s-1], each odd and
 *   below 2^k (e.g. the Joe-Kuo table; the rest of the row is not read).
 *   known [n] u8 device (nullable) = the admissibility of each row under the
 *   constraints (A, b, r) as scoot_known_constraints defines it, computed in
 *   the same pass.  poly, vinit, levels, A, b: host.  1 <= d <=
 *   SCOOT_MAX_DIM, 0 <= r <= SCOOT_MAX_CONSTRAINTS, skip >= 0, n >= 0,
 *   skip + n <= 2^32.
 *
 * scoot_known_constraints (device): known[i] = 1 when every row r of the
 *   linear constraints holds for row i of Xc [n*d] float32: sum over k = 0..d-1
 *   in order of A[r*d + k] * x_k, in double, each product and each partial sum
 *   rounded on its own, <= b[r]; else 0 (NaN inputs: 0).  A [r*d] and b [r]
 *   host, finite A, b not NaN.  Every rule the paper lists is such a row over
 *   the normalised knobs: an order between two knobs (x_a - x_b <= 0), "not
 *   both" booleans (x_a + x_b <= 1), "a implies b" (x_a - x_b <= 0), a bound
 *   that holds unless a boolean is set (big-M: c - x_a - M x_b <= 0).
 *
 * Errors: INVALID_ARG (null pointer, d out of range, negative level, bad
 * polynomial or initial number, non-finite A, NaN b, bad skip/n), UNSUPPORTED
 * (r or the polynomial degree beyond the limits), DEVICE.
 * ------------------------------------------------------------------------- */
int scoot_sobol_pool(const uint32_t* poly, const uint32_t* vinit, int d, const int32_t* levels, int64_t skip,
                     int64_t n, const double* A, const double* b, int r, float* Xc, uint8_t* known, void* stream);
int scoot_known_constraints(const float* Xc, int64_t n, int d, const double* A, const double* b, int r,
                            uint8_t* known, void* stream);

/* ---------------------------------------------------------------------------
 * The suggestion step, end to end (Algorithm 1, SUGGEST(k, O, RF, Delta); the
 * workflow of Sec. 4.1, steps 3-6): observed configurations and SLO values
 * in, k configurations to evaluate next out.  Host call; the device work runs
 * on `stream` and the call returns after it has finished.
 *
 * scoot_space: the search space.  levels [d] as in scoot_sobol_pool (0
 *   continuous, 1 boolean, L >= 2 a grid of L levels on [0, 1]); the Sobol
 *   direction tables sobol_poly [d] and sobol_vinit [d * SCOOT_SOBOL_MAX_DEGREE]
 *   as in scoot_sobol_pool; the known constraints A [r*d], b [r] (Sec. 4.5.3;
 *   r = 0: none, A and b may be NULL).
 *
 * scoot_suggest_opts: k (1 .. SCOOT_MAX_Q) configurations wanted; delta the
 *   POF threshold (Eq. 3, Algorithm 1); pool_size candidates (1 .. 2^31 - 1)
 *   starting at Sobol index pool_skip are scored (the solver's search);
 *   kernel and dtype of the GPs; warp_a, warp_b [p*d] (nullable, both or
 *   neither) fixed Kumaraswamy warps per objective; theta_lower,
 *   theta_upper, theta_start [p*(d+2)] (each nullable) the box and start of
 *   the maximum-likelihood search per objective in scoot_gp_mle's
 *   parameters, defaults: lengthscales [0.01, 10] from 0.5, signal variance
 *   [0.05, 20] from 1, noise variance [1e-6, 1] from 1e-3 (lower == upper
 *   fixes a parameter; all fixed skips the search); mle_max_iter (<= 0:
 *   200); n_trees (1 .. SCOOT_MAX_TREES), max_depth, forest_seed, bootstrap
 *   of the forest (scoot_forest_train); xi (Eq. 7-8); t >= 1 the tuning
 *   iteration of the UCB schedule and pick_seed of the random pick (one
 *   objective: MACE); ref [p] (nullable: worst valid observation + 10% of the
 *   range) the EHVI reference point in the caller's units (several
 *   objectives); learn_warp 1: the Kumaraswamy warping is learned with the
 *   other hyperparameters (scoot_gp_mle_warp; Sec. 4.3, the paper's
 *   Matern-3/2 with input warping), each warp parameter in [0.2, 5] starting
 *   from warp_a / warp_b when given, else from the identity a = b = 1; theta
 *   then has 3d + 2 entries per objective (theta_lower/upper/start keep their
 *   d + 2); 0: the warping is fixed (or absent) as given; host_search 0: the
 *   likelihood evaluations of the search run on the device
 *   (scoot_gp_mle_device, each objective on a stream of its own, the
 *   objectives side by side), 1: on the host (scoot_gp_mle).
 *
 * scoot_suggest: X_obs [n_obs*d] observed configurations (finite), Y_obs
 *   [n_obs*p] their objective values (minimised; read only where valid),
 *   valid [n_obs] 1 = the engine ran, 0 = it crashed (Sec. 4.7).  Steps:
 *   1. each objective's valid values are standardised (mean 0, standard
 *      deviation 1; a constant column keeps scale 1);
 *   2. per objective, hyperparameters by scoot_gp_mle from theta_start, then
 *      the GP by scoot_gp_fit_ex on the valid observations (prior mean 0);
 *   3. the forest by scoot_forest_train on every observation, label valid;
 *   4. the pool by scoot_sobol_pool with the known-constraint mask;
 *   5. one objective: scoot_suggest_mace_ex (best = the smallest valid
 *      standardised value, beta from scoot_ucb_beta(t)); several:
 *      scoot_score_pool_ex (EHVI over the valid standardised values, the
 *      reference point standardised alike), both under POF >= delta and the
 *      known constraints;
 *   6. a shortfall is filled with pool points in Sobol order that satisfy the
 *      known constraints and were not picked (Sec. 4.7, last paragraph); with
 *      no valid observation every suggestion comes from this fill (the
 *      initial design of Algorithm 1 is a call with n_obs = 0).
 *   x_out [k*d] host receives the configurations (the float32 pool points,
 *   widened), source [k] host (nullable) 0 = picked by the acquisition,
 *   1 = Sobol fill, theta_out [p*(d+2)], or [p*(3d+2)] with learn_warp, host
 *   (nullable) the hyperparameters used, *n_out the number written (below k only when the pool holds too
 *   few admissible points).  Library scratch on the current device holds the
 *   pool and the scores between calls.
 * Errors: INVALID_ARG (null pointer, bad sizes, non-finite input, p out of
 *   range, t < 1), UNSUPPORTED, NOT_PD, DEVICE, NO_MEMORY, and those of the
 *   calls made.
 * ------------------------------------------------------------------------- */
typedef struct scoot_space {
  int d;
  const int32_t* levels;
  const uint32_t* sobol_poly;
  const uint32_t* sobol_vinit;
  const double* A;
  const double* b;
  int r;
} scoot_space;

typedef struct scoot_suggest_opts {
  int k;
  double delta;
  int64_t pool_size;
  int64_t pool_skip;
  int kernel; /* scoot_kernel */
  int dtype;  /* scoot_dtype */
  const double* warp_a;
  const double* warp_b;
  const double* theta_lower;
  const double* theta_upper;
  const double* theta_start;
  int mle_max_iter;
  int n_trees;
  int max_depth;
  uint64_t forest_seed;
  int bootstrap;
  double xi;
  int t;
  uint64_t pick_seed;
  const double* ref;
  int learn_warp;
  int host_search;
} scoot_suggest_opts;

int scoot_suggest(const double* X_obs, const double* Y_obs, const uint8_t* valid, int n_obs, int p,
                  const scoot_space* space, const scoot_suggest_opts* opts, double* x_out, int32_t* source,
                  double* theta_out, int* n_out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SCOOT_H */
