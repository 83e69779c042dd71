/*
 * bart.h -- C ABI of libbart: the per-tree backfitting sweep of Bayesian
 * Additive Regression Trees (BART) on one AMD Instinct MI355X (gfx950).
 *
 * The method is the Metropolis-within-Gibbs sampler of "Very Fast Bayesian
 * Additive Regression Trees on GPU" (arXiv 2410.23244): sum-of-trees model
 * (sec. 2.1, eq. bartdef), GROW/PRUNE structure moves (sec. 3.3, "Tree
 * structure proposal"), exact leaf and error-variance draws (sec. 2.2 "The
 * BART MCMC", sec. 3.3), trees stored as fixed-size heaps (sec. 3.2) and an
 * index cache plus residual cache updated tree by tree (sec. 3.3).
 *
 * Conventions shared by every entry point:
 *  - D = max_depth, with D = 1 for a root-only tree (sec. 3.2); H = 2^(D-1).
 *    Heap index h >= 1, root 1, children 2h (left) and 2h+1 (right).
 *  - Tree arrays, one row per tree: axis u16 [ntree][H], cut u8 [ntree][H]
 *    (cut 0 = leaf, cuts start at 1), leaf f32 [ntree][2H].
 *  - X_b is the binned predictor matrix, predictor-major: u8 [p][x_stride],
 *    X_b[a][i] = index of observation i in the splitting grid of axis a, in
 *    [0, n_cuts[a]] (sec. 3.2, "Predictors").  Observation i goes right at
 *    node h iff X_b[axis[h]][i] >= cut[h] (Algorithm 1).
 *  - All device pointers are HIP device memory of the current device.  The
 *    library never allocates device memory: X_b and the workspace are
 *    borrowed from the caller and must outlive the handle.
 *  - Every call returns BART_OK (0) or a negative error code; arguments are
 *    validated before anything is enqueued, and on error nothing is enqueued
 *    and the state is unchanged.  bart_last_error() describes the last error
 *    of the calling thread.
 *  - Work is enqueued asynchronously on the handle's HIP stream; only
 *    bart_get_state() and bart_status() synchronise it.
 *  - A handle holds nchain >= 1 independent chains of the same model and
 *    data (sec. 2.2, "Behavior of the BART MCMC", advises running several
 *    and comparing them).  They share X_b and advance together, one sweep
 *    kernel launch serving all of them; each has its own trees, index cache,
 *    residuals, sigma^2 and random stream.
 */
#ifndef BART_H
#define BART_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BART_OK 0
#define BART_EINVAL (-1)   /* invalid argument or configuration */
#define BART_ENOSPACE (-2) /* workspace too small or misaligned */
#define BART_EHIP (-3)     /* a HIP runtime call failed */
#define BART_ESTATE (-4)   /* call not allowed in the handle's current state */
#define BART_ENOTSUP (-5)  /* size beyond what this build supports */
#define BART_EDEVICE (-6)  /* the device reported a failure (see bart_status) */

/* Device error bits reported by bart_status() */
#define BART_DEVERR_TIMEOUT 1u   /* a cross-workgroup wait exceeded its spin limit */
#define BART_DEVERR_CACHE 2u     /* index cache inconsistent with the trees */

/* How bart_step and bart_debug_steps launch the sweep kernel.  Its workgroups
 * wait on each other, so all of them must be resident at once.
 *  COOPERATIVE: hipLaunchCooperativeKernel, which guarantees co-residency.
 *  ORDINARY: hipLaunchKernel.  The grid never exceeds one workgroup per
 *    compute unit, so on a device with no other long-running work every
 *    workgroup becomes resident; kernels running concurrently on other
 *    streams only delay that, and a wait that outlasts its spin limit ends the
 *    launch with BART_DEVERR_TIMEOUT instead of hanging.  Use it where
 *    cooperative launches are unavailable (stream capture into a HIP graph,
 *    kernel tracers that cannot record them). */
#define BART_LAUNCH_COOPERATIVE 0
#define BART_LAUNCH_ORDINARY 1

/* Where the sweep kernel keeps the residual cache during a launch.
 *  REGISTERS: in the registers of the workgroups that own the observations,
 *    read at launch start and written back at launch end (up to about 4.2M
 *    observations on 256 compute units).
 *  STREAMED: in HBM, read and written once per tree step (any n).
 *  AUTO: registers when they fit, else streamed. */
#define BART_RESID_AUTO 0
#define BART_RESID_REGISTERS 1
#define BART_RESID_STREAMED 2

typedef struct bart_handle bart_handle;

/* Model and problem configuration. */
typedef struct {
  int32_t n;          /* observations, >= 1 */
  int32_t p;          /* predictors, >= 1 */
  int32_t ntree;      /* trees m (sec. 2.1 "Hyperparameters"), >= 1 */
  int32_t max_depth;  /* D in [2, 8]; nodes at depth D-1 are leaves */
  int32_t idx_bytes;  /* 1 or 2: width of the index cache entries; 0: no [ntree][n]
                         index cache (sec. 5, "Deeper limitations": it can be
                         dropped at some speed): every tree step routes the
                         observations by Algorithm 1 and two rolling u8 rows carry
                         a tree's leaves from the step that sums it to the step
                         that applies it; needs streamed residuals */
  int32_t grid;       /* workgroups of the sweep kernel per chain, each owning a
                         slice of the observations: 0 = automatic, else in
                         [1, 256] with grid x nchain <= compute units */
  int32_t launch;     /* BART_LAUNCH_COOPERATIVE or BART_LAUNCH_ORDINARY */
  int32_t residency;  /* BART_RESID_AUTO, BART_RESID_REGISTERS or BART_RESID_STREAMED */
  int32_t nchain;     /* independent chains: 0 or 1 = one, else in [1, 256] (at most
                         one per compute unit) */
  int32_t probit;     /* 0: regression; 1: binary y by the probit model (below) */
  int64_t x_stride;   /* elements between predictor rows of X_b: >= n, multiple of 16 */
  double alpha, beta; /* tree prior P_d = alpha (1+d)^-beta, alpha in [0,1], beta >= 0 */
  double mu_mu;       /* leaf prior mean (sec. 2.1 "Prior over leaf values") */
  double sigma_mu;    /* leaf prior sd, > 0 */
  double nu, lambda;  /* error-variance prior lambda nu / sigma^2 ~ chi^2_nu, > 0 */
  double sigma2_init; /* initial sigma^2, > 0 */
  double p_grow;      /* P(GROW) when both GROW and PRUNE are possible, in [0,1] */
  double probit_offset; /* probit: f(x) = probit_offset + sum of trees, finite */
} bart_config;

/* Probit model (binary outcomes, which the paper leaves to the BART
 * literature in sec. 5, "Mild limitations"): P(y = 1 | x) = Phi(f(x)), fitted
 * with latent z_i ~ N(f(x_i), 1), y_i = 1 iff z_i > 0 (Albert and Chib,
 * 1993).  bart_init reads y_i = [y_c[i] > 0], starts every latent at +-1 on
 * its side of 0 and the residuals at z_i - probit_offset; sigma^2 stays 1
 * (sigma2_init, nu and lambda are not used).  The step that ends a sweep
 * draws every z_i from N(f_i, 1) truncated to its side of 0, by inversion
 * of the normal cdf with one uniform per observation, and moves the residual
 * with it.  bart_predict gives f, to be passed through Phi. */

/* State of one chain, in the layouts above.  For bart_get_state the array
 * pointers are caller-owned device buffers that receive copies; for
 * bart_set_state they are read.  idx is dense [ntree][n] of idx_bytes-wide
 * entries (u8 when idx_bytes = 0: bart_get_state computes it by Algorithm 1
 * and bart_set_state ignores it).  chain selects the chain (input of both
 * calls). */
typedef struct {
  uint16_t *axis;
  uint8_t *cut;
  float *leaf;
  void *idx;
  float *resid;   /* [n]: y_c - sum of trees (sec. 3.3 "Residuals cache") */
  double sigma2;
  int64_t sweep;  /* index of the sweep in progress */
  int32_t next;   /* next step of that sweep: 0..ntree-1 trees, ntree = sigma^2 */
  int32_t chain;  /* in [0, nchain) */
  float *latent;  /* probit: [n] latents z_i (NULL: not copied); ignored otherwise */
  int32_t *count; /* bart_get_state only: per-leaf counts i32 [ntree][2H] the sampler
                     keeps (slot h, a leaf: observations in it; other slots hold
                     stale values nothing reads), NULL: not copied; bart_set_state
                     ignores it and recounts from idx */
} bart_state;

/* Per-step record written by bart_debug_steps (4224 bytes).  Slots are heap
 * indices; count/sum cover the leaves of the larger tree of the move (the
 * proposed tree for GROW, the current tree for PRUNE, sec. 3.3 "Traverse
 * indices cache"), leaf_new the leaves of the final tree. */
typedef struct {
  int32_t kind;      /* 0 tree step, 1 sigma^2 step */
  int32_t tree;
  int64_t sweep;
  int32_t move;      /* 0 none, 1 GROW, 2 PRUNE */
  int32_t eta, axis, cut;
  int32_t n_grow_cand, n_prune_cand; /* #growable leaves, #prunable nodes of T */
  int32_t accept;
  int32_t n_leaves;
  double log_r, ln_u;
  double log_r_scale;  /* unused on the device (0) */
  double ssr, sigma2;  /* sigma^2 step: sum of squared residuals and new sigma^2 */
  int32_t pad[10];
  int32_t count[256];
  double sum[256];     /* partial-residual sums S_h = sum r_i + n_h * old value */
  float leaf_new[256];
} bart_trace;

/* Launch shape chosen by bart_init (grid: workgroups per chain; the launch
 * has grid x nchain workgroups).  rank_stash: 1 if streamed residuals keep
 * each tree's leaf ranks in LDS from the pass that accumulates the tree to
 * the pass that applies its decision (a thread's chunks fit the stash), 0
 * otherwise.  stash_chunks: the most chunks of 4 observations per thread the
 * stash holds.  lds_resid_chunks: with the stash, how many of a thread's
 * chunks keep their residuals in LDS for the whole launch (the others stream
 * from HBM every tree step); 0 otherwise. */
typedef struct {
  int32_t grid, block, chunks_per_thread, lds_bytes;
  int32_t obs_per_thread, max_leaves, launch, residency;
  int32_t nchain, rank_stash, stash_chunks, lds_resid_chunks;
} bart_launch;

/* Bytes of device workspace bart_init needs for cfg (0 if cfg is invalid). */
size_t bart_workspace_bytes(const bart_config *cfg);

/* Create nchain chains.  X_b: device u8 [p][x_stride], borrowed.  y_c: device
 * f32 [n], the centred response, copied into every chain's residual cache.  n_cuts: HOST
 * int32 [p], number of cutpoints K_a in [0, 255] of each axis, copied.
 * workspace: device, >= bart_workspace_bytes(cfg), 256-byte aligned,
 * borrowed.  stream: a hipStream_t (NULL = default stream).  Initial state of
 * every chain: every tree root-only with leaf 0, index cache 1, residuals =
 * y_c, sigma^2 = sigma2_init, sweep 0 (sec. 3.3 "Residuals cache").  On
 * success *out receives the handle. */
int bart_init(const bart_config *cfg, const uint8_t *X_b, const float *y_c,
              const int32_t *n_cuts, void *workspace, size_t ws_bytes, void *stream,
              bart_handle **out);

/* Run k_sweeps >= 0 whole sweeps of every chain (each: every tree in order,
 * then sigma^2; sec. 2.2 "The BART MCMC").  The chains must be at a sweep
 * boundary (BART_ESTATE otherwise).  Random draws of chain c, sweep s, tree j
 * are a pure function of (seed, c, s, j): Philox4x64-10 with key (seed,
 * 0x42415254) and counter (s, j, q, c 2^32 + t), the chain offset in counter
 * word 3 (q selects the proposal block, the leaf normals or the sigma^2
 * gamma attempts, t the slot pair or attempt, always below 2^32), so chain 0
 * draws what a lone chain draws, no two chains share a counter, and two
 * calls of k sweeps equal one call of 2k. */
int bart_step(bart_handle *h, int32_t k_sweeps, uint64_t seed);

/* For callers that cannot allocate device memory or must not have the
 * library touch caller memory beyond the handle's state (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * sweeps as bart_step, with the same arguments, results and error behaviour,
 * but the sweep kernel's cross-workgroup mailboxes (its only scratch data:
 * per-workgroup partial sums tagged with step numbers) live in a static
 * device array of the library instead of the workspace.  The array holds 2 x
 * 256 x 144 64-bit words (576 KiB) per device, enough for every launch shape
 * bart_init accepts (grid x nchain <= 256 workgroups); it is held by each
 * device the library runs on until the process ends.  The call allocates
 * nothing and enqueues only kernels (a fill kernel clears the mailboxes at
 * the start of every launch, so contents left by earlier calls are never
 * read).  All calls on one device share that array: calls that overlap on
 * one device (handles driven from different streams or threads at the same
 * time) race and produce wrong results; calls ordered on one stream, or
 * separated by synchronisation, are safe.  BART_ENOTSUP if the handle's
 * mailboxes would not fit the array. */
int bart_step_static(bart_handle *h, int32_t k_sweeps, uint64_t seed);

/* Add f(x) and f(x)^2, in fp64 before rounding, to sum and sumsq (device
 * f64 [nchain][n_t]) for every chain: called once per kept sweep it
 * accumulates the posterior mean and variance of f at the points of Xt
 * (sec. 2.2: the samples of the chain approximate the posterior).  Xt as
 * for bart_predict. */
int bart_predict_accumulate(bart_handle *h, const uint8_t *Xt, int64_t xt_stride, int64_t n_t,
                            double offset, double *sum, double *sumsq);

/* Posterior mean and sd of f at n_t points from the sums that
 * bart_predict_accumulate gathered over n_keep kept sweeps of every chain
 * (sec. 2.2: the kept samples of the chains approximate the posterior; the
 * chains are pooled).  Per point, chain c's mean m_c = sum[c] / n_keep and
 * variance v_c = sumsq[c] / n_keep - m_c^2; mean = the average of the m_c;
 * sd = sqrt(max(0, average of the v_c + variance of the m_c over the
 * chains)), the law of total variance.  sum, sumsq: device f64
 * [nchain][n_t]; mean, sd: device f64 [n_t]. */
int bart_posterior_summary(bart_handle *h, const double *sum, const double *sumsq, int64_t n_t,
                           int64_t n_keep, double *mean, double *sd);

/* Sum-of-trees prediction f(x) = offset + sum_j g(x; T_j, M_j) (eq. bartdef),
 * each tree traversed by Algorithm 1, summed in fp64 in tree order and
 * rounded to f32, for every chain.  Xt: device u8 [p][xt_stride] binned like
 * X_b, xt_stride >= n_t and a multiple of 16; out: device f32 [nchain][n_t]. */
int bart_predict(bart_handle *h, const uint8_t *Xt, int64_t xt_stride, int64_t n_t,
                 double offset, float *out);

/* Copy the state of chain dst->chain into caller device buffers and fill
 * the scalars; this synchronises the handle's stream.  A NULL array pointer
 * skips that array (all NULL: only sigma^2 and the position). */
int bart_get_state(bart_handle *h, bart_state *dst);

/* Replace the state of chain src->chain from caller device buffers (index
 * cache and trees must be consistent: every idx entry a leaf of its tree).
 * Per-leaf counts are recomputed on the device; an idx entry outside heap
 * slots 1..2H-1 sets BART_DEVERR_CACHE (reported by bart_status), and a
 * leaf index that is not a leaf of its tree does so during the next
 * sweep.  The position (sweep, next) is shared by all chains: setting it
 * moves every chain. */
int bart_set_state(bart_handle *h, const bart_state *src);

/* Run the next n_steps steps (tree steps and sigma^2 steps, in order, from
 * any position) with the same kernel as bart_step, writing one record per
 * step and chain into trace (device bart_trace [nchain][n_steps]). */
int bart_debug_steps(bart_handle *h, int32_t n_steps, uint64_t seed, bart_trace *trace);

/* Test hook for the bounded waits: one launch of n_steps steps (1 ..
 * 2^20 - 8) in which workgroup wg of the launch grid (0 <= wg < grid x
 * nchain) returns at once and every cross-workgroup wait gives up after
 * spin_limit (>= 1) poll rounds.  Every other workgroup of wg's chain then
 * ends the launch and bart_status reports BART_DEVERR_TIMEOUT.  The chains'
 * state afterwards is unspecified (only bart_set_state or bart_destroy are
 * meaningful); the position does not move.  With one workgroup per chain
 * there is no cross-workgroup wait and nothing times out. */
int bart_debug_stall(bart_handle *h, int32_t n_steps, uint64_t seed, int32_t wg,
                     uint32_t spin_limit);

/* Synchronise the stream and return BART_OK, or BART_EDEVICE with the device
 * error bits of all chains (or-ed) in *bits (may be NULL). */
int bart_status(bart_handle *h, uint32_t *bits);

/* Move statistics of one chain since bart_init (sec. 2.2, "Behavior of the
 * BART MCMC": acceptance is typically 10-30 %, trees stay small): out[0]
 * GROW proposed, out[1] PRUNE proposed, out[2] GROW accepted, out[3] PRUNE
 * accepted, out[4] tree steps, out[5] the sum over tree steps of the leaves
 * of the tree after the step.  Synchronises the handle's stream. */
int bart_move_stats(bart_handle *h, int32_t chain, uint64_t *out);

/* Launch shape of the sweep kernel. */
int bart_launch_info(const bart_handle *h, bart_launch *out);

/* ---- Host-side preparation (no device, no handle; sec. 3.2 "Predictors",
 * sec. 2.1 "Hyperparameters").  Host arrays, row-major by predictor. */

#define BART_GRID_UNIFORM 0  /* K cuts evenly spaced strictly inside [min, max] */
#define BART_GRID_QUANTILE 1 /* K empirical quantiles at k/(K+1), k = 1..K */

/* Splitting grid of every predictor.  X: host f32 [p][ldx] (finite), K in
 * [1, 255] cuts per predictor.  UNIFORM: c_k = min + k (max - min)/(K+1).
 * QUANTILE: linear interpolation between order statistics at position
 * (n - 1) k/(K+1).  Repeated cuts, and quantile cuts at the minimum, are
 * dropped, so n_cuts[a] <= K; a constant predictor gets none.  cuts: host
 * f64 [p][K], increasing in its first n_cuts[a] entries, +inf after. */
int bart_cutpoints(const float *X, int64_t n, int32_t p, int64_t ldx, int32_t K, int32_t grid,
                   double *cuts, int32_t *n_cuts);

/* Binned predictors X_b[a][i] = #{k < n_cuts[a] : cuts[a][k] <= X[a][i]}
 * (0 for NaN), so that "right iff X_b >= s" means "X >= c_s".  X: host f32
 * [p][ldx]; cuts/n_cuts as from bart_cutpoints (row stride K); X_b: host u8
 * [p][ldb], columns [0, n) written. */
int bart_bin(const float *X, int64_t n, int32_t p, int64_t ldx, const double *cuts,
             const int32_t *n_cuts, int32_t K, uint8_t *X_b, int64_t ldb);

/* Default hyperparameters from the response y (host f64 [n]): offset =
 * mean(y); y_c = f32(y - offset) (host [n]); in cfg: alpha 0.95, beta 2,
 * mu_mu 0, sigma_mu = (max - min of y_c) / (4 sqrt(ntree)) (the data range
 * at +-2 prior sd of the sum of trees), nu 3, lambda = var(y) q / nu with q
 * the 0.1 quantile of chi^2_nu (the data variance at the 0.9 prior
 * quantile of sigma^2), sigma2_init = var(y), p_grow 0.5.  Other fields of
 * cfg are left as they are. */
int bart_default_hyper(const double *y, int64_t n, int32_t ntree, double *offset, float *y_c,
                       bart_config *cfg);

/* Release the handle (the caller frees X_b and the workspace). */
void bart_destroy(bart_handle *h);

/* Message of the last error on the calling thread ("" if none). */
const char *bart_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* BART_H */
