/*
 * bart_oracle.h -- plain CPU reference ("oracle") of the BART
 * Metropolis-within-Gibbs sweep of "Very Fast Bayesian Additive Regression
 * Trees on GPU" (arXiv 2410.23244).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  The product path
 * (the HIP library) never includes, links or calls anything in oracle/.
 * It shares no source with the HIP path: its random generator, samplers,
 * tree bookkeeping and arithmetic are written here from the paper and the
 * published definitions they cite.
 *
 * Conventions (paper sec. 3.2 "Representation of variables"):
 *   heap index h >= 1, root = 1, children 2h (left) and 2h+1 (right);
 *   D = maximum depth with D = 1 for a root-only tree;
 *   H = 2^(D-1): axis[] and cut[] have H entries (nodes at depth D-1 are
 *   always leaves), leaf[] has 2H entries; cut 0 marks a leaf and cuts
 *   start from 1.  Observation i goes right at node h iff
 *   X[axis[h]][i] >= cut[h] (Algorithm 1).
 * Storage types match the device state so states exchange bit-exactly:
 *   axis u16, cut u8, leaf f32, idx u8 or u16, residual f32, sigma^2 f64.
 */
#ifndef BART_ORACLE_H
#define BART_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t n, p, m, D, idx_bytes;  /* observations, predictors, trees, depth, 1|2 */
  int32_t fix_sigma2;             /* test hook: 1 = keep sigma^2 fixed (no Gibbs draw) */
  int32_t chain;                  /* which chain's random stream (>= 0) */
  int32_t pad;
  double alpha, beta;             /* tree prior P_d = alpha/(1+d)^beta (sec. 2.1) */
  double mu_mu, sigma_mu;         /* leaf prior N(mu_mu, sigma_mu^2) (sec. 2.1) */
  double nu, lambda;              /* lambda*nu/sigma^2 ~ chi^2_nu (eq. bartdef) */
  double p_grow;                  /* P(GROW) when both moves are possible */
  int32_t probit;                 /* 1: binary y, latent-variable probit model */
  int32_t pad2;
  double probit_offset;           /* probit: f(x) = offset + sum of trees */
} oc_config;

/* Mutable chain state.  All arrays are caller-owned. */
typedef struct {
  uint16_t *axis;   /* [m][H] */
  uint8_t *cut;     /* [m][H] */
  float *leaf;      /* [m][2H] */
  void *idx;        /* [m][n] u8 or u16: leaf of each observation per tree */
  float *resid;     /* [n]: full residuals y - sum of trees */
  double sigma2;
  int64_t sweep;    /* index s of the sweep in progress */
  int32_t next;     /* next step of sweep s: 0..m-1 tree steps, m = sigma^2 step */
  float *latent;    /* probit: [n] latent z_i (y_i = 1 iff z_i > 0) */
  const uint8_t *ybin; /* probit: [n] binary response */
} oc_state;

/* Per-step trace record (4224 bytes). */
typedef struct {
  int32_t kind;       /* 0 tree step, 1 sigma^2 step */
  int32_t tree;
  int64_t sweep;
  int32_t move;       /* 0 none, 1 grow, 2 prune */
  int32_t eta, axis, cut;
  int32_t n_grow_cand, n_prune_cand;   /* #G(T), #P(T) */
  int32_t accept;
  int32_t n_leaves;   /* leaves of the larger tree of the move */
  double log_r, ln_u;
  double log_r_scale; /* sum of |terms| of log r (tie band) */
  double ssr, sigma2; /* sigma^2 step only */
  int32_t pad[10];
  int32_t count[256]; /* per heap slot, leaves of the larger tree */
  double sum[256];    /* partial-residual sums S_h, same slots */
  float leaf_new[256];/* new leaf values at the leaves of the final tree */
} oc_trace;

void oc_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]);
double oc_norm_cdf(double x);
double oc_norm_ppf(double p);
double oc_latent_draw(double f, int32_t y, double u);
double oc_normal(uint64_t seed, uint64_t s, uint64_t j, uint64_t slot);
double oc_sigma2_draw(uint64_t seed, uint64_t s, double nu, double lambda, int64_t n,
                      double ssr);
double oc_gamma_draw(uint64_t seed, uint64_t s, double shape);

int oc_tree_info(const oc_config *c, const int32_t *n_cuts, const uint16_t *axis,
                 const uint8_t *cut, int32_t *is_leaf, int32_t *p_adj, double *p_split,
                 int32_t *grow_list, int32_t *n_grow, int32_t *prune_list, int32_t *n_prune);
double oc_log_prior(const oc_config *c, const int32_t *n_cuts, const uint16_t *axis,
                    const uint8_t *cut);
void oc_propose(const oc_config *c, const int32_t *n_cuts, const uint16_t *axis,
                const uint8_t *cut, const uint64_t words[4], int32_t out[6]);
double oc_llr(double sigma2, double mu_mu, double sigma_mu, double nL, double SL,
              double nR, double SR);
void oc_leaf_posterior(double n, double S, double sigma2, double mu_mu, double sigma_mu,
                       double *mean, double *prec);
double oc_log_ratio(const oc_config *c, const int32_t *n_cuts, const uint8_t *X,
                    int64_t ldx, const uint16_t *axis, const uint8_t *cut, const float *leaf,
                    const void *idx_row, const float *resid, double sigma2, int32_t move,
                    int32_t eta, int32_t a, int32_t s, double *scale);
int32_t oc_route(int32_t D, const uint16_t *axis, const uint8_t *cut, const uint8_t *X,
                 int64_t ldx, int64_t i);
/* oc_normal, oc_gamma_draw and oc_sigma2_draw draw from chain 0's stream.
 * One step (tree step `next`, or the sigma^2 step) of chain c->chain.  Lockstep hooks for
 * comparing another implementation step by step: force >= 0 replaces the
 * accept decision of a tree step; adopt (256 floats, or NULL) replaces the
 * new leaf values used to update the state after they were drawn and
 * recorded in the trace.  Neither changes what the trace reports. */
int oc_step(const oc_config *c, const int32_t *n_cuts, const uint8_t *X, int64_t ldx,
            oc_state *st, uint64_t seed, int32_t force, const float *adopt, oc_trace *trace);
int oc_run(const oc_config *c, const int32_t *n_cuts, const uint8_t *X, int64_t ldx,
           oc_state *st, uint64_t seed, int64_t n_steps, oc_trace *traces);
void oc_predict(const oc_config *c, const uint16_t *axis, const uint8_t *cut,
                const float *leaf, const uint8_t *Xt, int64_t ldxt, int64_t nt,
                double offset, float *out);

#ifdef __cplusplus
}
#endif
#endif
