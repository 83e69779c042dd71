/*
 * bart_oracle.c -- plain, slow, scalar CPU reference of the BART sweep of
 * "Very Fast Bayesian Additive Regression Trees on GPU" (arXiv 2410.23244).
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the tests, the smoke check and the
 * CPU-baseline leg of the benchmark, never by the product path.
 *
 * The method (paper sec. 2.1-2.2 and sec. 3.3): the sum-of-trees model of
 * eq. (bartdef) with the tree prior of sec. 2.1 and a fixed maximum depth
 * (sec. 3.1, 3.2); each sweep updates the trees in order with a GROW/PRUNE
 * Metropolis-Hastings step on the structure (sec. 3.3 "Tree structure
 * proposal"), an exact draw of the leaves, a residual-cache update
 * (sec. 3.3 "Residuals cache"), then an exact draw of sigma^2 (sec. 3.3
 * "Sampling the error variance").  The paper does not print the MH ratio;
 * it is derived here from the priors of sec. 2.1 and the GROW/PRUNE
 * proposal, and pinned by exact enumeration in the tests.
 *
 * Everything is computed one observation at a time, in index order, with
 * fp64 accumulation; residuals and leaf values are stored in fp32, as the
 * paper does (app. B, "Numerical error due to caching residuals").
 */
#include "bart_oracle.h"

#include <float.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

#ifndef M_PI
#define M_PI 3.14159265358979323846
#endif
#ifndef M_SQRT1_2
#define M_SQRT1_2 0.70710678118654752440
#endif

/* ------------------------------------------------------------------ */
/* Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11), from its published
 * definition: 10 rounds of two 64x64->128 multiplies with a Weyl key
 * schedule.  The paper pre-generates its random numbers as uniforms and
 * normals (sec. 3.3 "Generate random samples"); a counter-based generator
 * makes every draw a pure function of (seed, sweep, tree, slot).         */

static const uint64_t PH_M0 = 0xD2E7470EE14C6C93ULL;
static const uint64_t PH_M1 = 0xCA5A826395121157ULL;
static const uint64_t PH_W0 = 0x9E3779B97F4A7C15ULL;
static const uint64_t PH_W1 = 0xBB67AE8584CAA73BULL;
static const uint64_t KEY_TAG = 0x42415254ULL; /* second key word */

void oc_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]) {
  uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint64_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; round++) {
    if (round > 0) {
      k0 += PH_W0;
      k1 += PH_W1;
    }
    unsigned __int128 p0 = (unsigned __int128)PH_M0 * x0;
    unsigned __int128 p1 = (unsigned __int128)PH_M1 * x2;
    uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
    uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    x0 = hi1 ^ x1 ^ k0;
    x1 = lo1;
    x2 = hi0 ^ x3 ^ k1;
    x3 = lo0;
  }
  out[0] = x0;
  out[1] = x1;
  out[2] = x2;
  out[3] = x3;
}

/* Stream layout of chain c: counter (s, j, q, c 2^32 + t), key (seed,
 * "BART"); every t is below 2^32, so no two chains share a counter and
 * chain 0 is the stream of a lone chain.
 *   q = 0, t = 0     proposal words of tree j in sweep s
 *   q = 1, t = h>>1  the two leaf normals of heap slots 2t, 2t+1
 *   q = 2, j = ~0    sigma^2 gamma attempts t = 0, 1, ...            */
static void block(uint64_t seed, uint32_t chain, uint64_t s, uint64_t j, uint64_t q,
                  uint64_t t, uint64_t out[4]) {
  uint64_t ctr[4] = {s, j, q, ((uint64_t)chain << 32) + t};
  uint64_t key[2] = {seed, KEY_TAG};
  oc_philox4x64_10(ctr, key, out);
}

/* uniform strictly inside (0,1): (k + 1/2) 2^-52 with k the top 52 bits of
 * w; every such value is exact in fp64 (k + 1/2 needs 53 bits) */
static double u01(uint64_t w) { return ((double)(w >> 12) + 0.5) * 0x1.0p-52; }

/* integer in [0, k) by multiply-shift of a 32-bit word (Lemire 2019,
 * without the rejection step) */
static int32_t pick(uint32_t w, int32_t k) {
  return (int32_t)(((uint64_t)w * (uint64_t)(uint32_t)k) >> 32);
}

/* Box-Muller (1958), cosine branch */
static double box_muller(uint64_t w_a, uint64_t w_b) {
  double u1 = u01(w_a), u2 = u01(w_b);
  return sqrt(-2.0 * log(u1)) * cos(2.0 * M_PI * u2);
}

static double normal_of(uint64_t seed, uint32_t chain, uint64_t s, uint64_t j, uint64_t slot) {
  uint64_t w[4];
  block(seed, chain, s, j, 1, slot >> 1, w);
  return (slot & 1) ? box_muller(w[2], w[3]) : box_muller(w[0], w[1]);
}

double oc_normal(uint64_t seed, uint64_t s, uint64_t j, uint64_t slot) {
  return normal_of(seed, 0, s, j, slot);
}

/* Gamma(shape, 1) by Marsaglia & Tsang (2000), shape >= 1. */
static double gamma_of(uint64_t seed, uint32_t chain, uint64_t s, double shape) {
  double d = shape - 1.0 / 3.0;
  double c = 1.0 / sqrt(9.0 * d);
  for (uint64_t t = 0; t < 4096; t++) {
    uint64_t w[4];
    block(seed, chain, s, ~0ULL, 2, t, w);
    double z = box_muller(w[0], w[1]);
    double u = u01(w[2]);
    double v = 1.0 + c * z;
    v = v * v * v;
    if (v > 0.0 && log(u) < 0.5 * z * z + d - d * v + d * log(v)) return d * v;
  }
  return d;
}

/* sigma^2 | rest ~ InvGamma((nu+n)/2, (nu*lambda + SSR)/2): the prior
 * lambda*nu/sigma^2 ~ chi^2_nu of eq. (bartdef) is InvGamma(nu/2,
 * nu*lambda/2), conjugate to the normal errors (sec. 3.3 "Sampling the
 * error variance"). */
double oc_gamma_draw(uint64_t seed, uint64_t s, double shape) {
  return gamma_of(seed, 0, s, shape);
}

static double sigma2_of(uint64_t seed, uint32_t chain, uint64_t s, double nu, double lambda,
                        int64_t n, double ssr) {
  double shape = 0.5 * (nu + (double)n);
  double scale = 0.5 * (nu * lambda + ssr);
  return scale / gamma_of(seed, chain, s, shape);
}

double oc_sigma2_draw(uint64_t seed, uint64_t s, double nu, double lambda, int64_t n,
                      double ssr) {
  return sigma2_of(seed, 0, s, nu, lambda, n, ssr);
}

/* ------------------------------------------------------------------ */
/* Probit model for binary y (sec. 5, "Mild limitations": binary outcomes
 * follow the BART literature), by the latent-variable augmentation of
 * Albert and Chib (1993): z_i ~ N(f(x_i), 1), y_i = 1 iff z_i > 0, so given
 * the trees z_i is a normal truncated to the side its y_i fixes, and given
 * the z_i the trees are fitted to z with sigma^2 = 1.                   */

double oc_norm_cdf(double x) { return 0.5 * erfc(-x * M_SQRT1_2); }

/* Inverse of oc_norm_cdf.  Solved in the lower tail, where the cdf is
 * accurate, for q = min(p, 1 - p) (1 - p is exact for p >= 1/2) and
 * reflected: a start from the rational approximation of Abramowitz and
 * Stegun 26.2.23 (|error| < 4.5e-4), then Newton steps on oc_norm_cdf until
 * they stop moving the root. */
double oc_norm_ppf(double p) {
  if (!(p > 0.0)) return -INFINITY;
  if (!(p < 1.0)) return INFINITY;
  double q = p < 0.5 ? p : 1.0 - p;
  double t = sqrt(-2.0 * log(q));
  double x = -(t - (2.515517 + 0.802853 * t + 0.010328 * t * t) /
                       (1.0 + 1.432788 * t + 0.189269 * t * t + 0.001308 * t * t * t));
  for (int it = 0; it < 50; it++) {
    double dens = exp(-0.5 * x * x) / sqrt(2.0 * M_PI);
    double dx = (oc_norm_cdf(x) - q) / dens;
    x -= dx;
    if (fabs(dx) <= 1e-15 * (1.0 + fabs(x))) break;
  }
  return p < 0.5 ? x : -x;
}

/* z | f, y ~ N(f, 1) truncated to z > 0 (y = 1) or z <= 0 (y = 0), by
 * inversion on the allowed side: with e = z - f, P(e < -f) = Phi(-f), so
 * y = 0 takes e = Phi^-1(u Phi(-f)) and y = 1 takes e = -Phi^-1(u Phi(f)). */
double oc_latent_draw(double f, int32_t y, double u) {
  double p = u * oc_norm_cdf(y ? f : -f);
  if (p < 1e-300) p = 1e-300;
  return y ? f - oc_norm_ppf(p) : f + oc_norm_ppf(p);
}

/* ------------------------------------------------------------------ */
/* Tree bookkeeping on the heap (sec. 3.2), by plain enumeration.       */

static int depth_of(int32_t h) {
  int d = 0;
  while (h > 1) {
    h >>= 1;
    d++;
  }
  return d;
}

static int present(const uint8_t *cut, int32_t h) {
  while (h > 1) {
    int32_t q = h >> 1;
    if (cut[q] == 0) return 0;
    h = q;
  }
  return 1;
}

static int is_leaf_node(const uint8_t *cut, int32_t H, int32_t h) {
  return present(cut, h) && (h >= H || cut[h] == 0);
}

/* Region of node h on every axis: cut indices lo[a]..hi[a] in [0, K_a].
 * The available splitting points of h on axis a are lo[a]+1 .. hi[a]
 * (sec. 2.1 "Prior over tree structure"). */
static void region(int32_t p, const int32_t *n_cuts, const uint16_t *axis,
                   const uint8_t *cut, int32_t h, int32_t *lo, int32_t *hi) {
  for (int32_t a = 0; a < p; a++) {
    lo[a] = 0;
    hi[a] = n_cuts[a];
  }
  int d = depth_of(h);
  for (int k = d; k >= 1; k--) {
    int32_t q = h >> k;          /* ancestor */
    int32_t child = h >> (k - 1);
    int32_t a = axis[q], s = cut[q];
    if (child & 1)
      lo[a] = s;                 /* right: x >= s */
    else
      hi[a] = s - 1;             /* left: x <= s-1 */
  }
}

static int32_t count_avail_axes(int32_t p, const int32_t *lo, const int32_t *hi) {
  int32_t k = 0;
  for (int32_t a = 0; a < p; a++)
    if (hi[a] - lo[a] > 0) k++;
  return k;
}

/* P_split(h) = alpha (1+d)^-beta if h may split, else 0 (sec. 2.1), with
 * the fixed maximum depth: nodes at depth D-1 are leaves (sec. 3.1, app. B). */
static double psplit(const oc_config *c, int32_t h, int32_t padj) {
  int d = depth_of(h);
  if (d >= c->D - 1 || padj <= 0) return 0.0;
  return c->alpha * pow(1.0 + (double)d, -c->beta);
}

typedef struct {
  int32_t *lo, *hi;
} scratch;

static double psplit_of(const oc_config *c, const int32_t *n_cuts, const uint16_t *axis,
                        const uint8_t *cut, int32_t h, scratch *sc) {
  region(c->p, n_cuts, axis, cut, h, sc->lo, sc->hi);
  return psplit(c, h, count_avail_axes(c->p, sc->lo, sc->hi));
}

/* G(T): growable leaves (P_split > 0), P(T): internal nodes whose two
 * children are leaves; both in increasing heap order. */
static void move_lists(const oc_config *c, const int32_t *n_cuts, const uint16_t *axis,
                       const uint8_t *cut, int32_t *G, int32_t *nG, int32_t *P,
                       int32_t *nP, scratch *sc) {
  int32_t H = 1 << (c->D - 1);
  *nG = 0;
  *nP = 0;
  for (int32_t h = 1; h < 2 * H; h++) {
    if (is_leaf_node(cut, H, h)) {
      if (psplit_of(c, n_cuts, axis, cut, h, sc) > 0.0) G[(*nG)++] = h;
    } else if (h < H && present(cut, h)) {
      if (is_leaf_node(cut, H, 2 * h) && is_leaf_node(cut, H, 2 * h + 1)) P[(*nP)++] = h;
    }
  }
}

static double prob_grow(const oc_config *c, int32_t nG, int32_t nP) {
  if (nP == 0) return 1.0;
  if (nG == 0) return 0.0;
  return c->p_grow;
}

int oc_tree_info(const oc_config *c, const int32_t *n_cuts, const uint16_t *axis,
                 const uint8_t *cut, int32_t *is_leaf, int32_t *p_adj, double *p_split,
                 int32_t *grow_list, int32_t *n_grow, int32_t *prune_list, int32_t *n_prune) {
  int32_t H = 1 << (c->D - 1);
  scratch sc = {malloc(sizeof(int32_t) * c->p), malloc(sizeof(int32_t) * c->p)};
  for (int32_t h = 0; h < 2 * H; h++) {
    is_leaf[h] = 0;
    p_adj[h] = 0;
    p_split[h] = 0.0;
    if (h == 0 || !present(cut, h)) continue;
    is_leaf[h] = is_leaf_node(cut, H, h);
    region(c->p, n_cuts, axis, cut, h, sc.lo, sc.hi);
    p_adj[h] = count_avail_axes(c->p, sc.lo, sc.hi);
    p_split[h] = psplit(c, h, p_adj[h]);
  }
  move_lists(c, n_cuts, axis, cut, grow_list, n_grow, prune_list, n_prune, &sc);
  free(sc.lo);
  free(sc.hi);
  return 0;
}

/* log pi(T): product over internal nodes of P_split/(p_adj * avail(axis)),
 * times product over leaves of (1 - P_split) (sec. 2.1). */
double oc_log_prior(const oc_config *c, const int32_t *n_cuts, const uint16_t *axis,
                    const uint8_t *cut) {
  int32_t H = 1 << (c->D - 1);
  scratch sc = {malloc(sizeof(int32_t) * c->p), malloc(sizeof(int32_t) * c->p)};
  double lp = 0.0;
  for (int32_t h = 1; h < 2 * H; h++) {
    if (!present(cut, h)) continue;
    region(c->p, n_cuts, axis, cut, h, sc.lo, sc.hi);
    int32_t padj = count_avail_axes(c->p, sc.lo, sc.hi);
    double ps = psplit(c, h, padj);
    if (is_leaf_node(cut, H, h)) {
      lp += log(1.0 - ps);
    } else {
      int32_t a = axis[h];
      lp += log(ps) - log((double)padj) - log((double)(sc.hi[a] - sc.lo[a]));
    }
  }
  free(sc.lo);
  free(sc.hi);
  return lp;
}

/* Proposal of sec. 3.3 (GROW and PRUNE only): from the four proposal words
 * w0..w3 of (s, j).  out = {move, eta, axis, cut, #G(T), #P(T)}. */
void oc_propose(const oc_config *c, const int32_t *n_cuts, const uint16_t *axis,
                const uint8_t *cut, const uint64_t w[4], int32_t out[6]) {
  int32_t H = 1 << (c->D - 1);
  int32_t *G = malloc(sizeof(int32_t) * 2 * H), *P = malloc(sizeof(int32_t) * 2 * H);
  scratch sc = {malloc(sizeof(int32_t) * c->p), malloc(sizeof(int32_t) * c->p)};
  int32_t nG, nP;
  move_lists(c, n_cuts, axis, cut, G, &nG, P, &nP, &sc);
  int32_t move = 0, eta = 0, a = 0, s = 0;
  if (nG > 0 || nP > 0) {
    double pg = prob_grow(c, nG, nP);
    if (u01(w[0]) < pg) {
      move = 1;
      eta = G[pick((uint32_t)w[1], nG)];
      region(c->p, n_cuts, axis, cut, eta, sc.lo, sc.hi);
      int32_t padj = count_avail_axes(c->p, sc.lo, sc.hi);
      int32_t k = pick((uint32_t)(w[1] >> 32), padj);
      for (int32_t b = 0; b < c->p; b++) {
        if (sc.hi[b] - sc.lo[b] > 0) {
          if (k == 0) {
            a = b;
            break;
          }
          k--;
        }
      }
      s = sc.lo[a] + 1 + pick((uint32_t)w[2], sc.hi[a] - sc.lo[a]);
    } else {
      move = 2;
      eta = P[pick((uint32_t)w[1], nP)];
    }
  }
  out[0] = move;
  out[1] = eta;
  out[2] = a;
  out[3] = s;
  out[4] = nG;
  out[5] = nP;
  free(G);
  free(P);
  free(sc.lo);
  free(sc.hi);
}

/* Log marginal-likelihood ratio of splitting a leaf into (L, R): the
 * partial residuals of a leaf with n points are N(mu_mu 1, sigma^2 I +
 * sigma_mu^2 1 1^T) once the N(mu_mu, sigma_mu^2) leaf (sec. 2.1) is
 * integrated out. */
double oc_llr(double sigma2, double mu_mu, double sigma_mu, double nL, double SL, double nR,
              double SR) {
  double v = sigma_mu * sigma_mu;
  double nP = nL + nR, SP = SL + SR;
  double tL = SL - nL * mu_mu, tR = SR - nR * mu_mu, tP = SP - nP * mu_mu;
  double QL = tL * tL / (sigma2 + nL * v);
  double QR = tR * tR / (sigma2 + nR * v);
  double QP = tP * tP / (sigma2 + nP * v);
  double det = 0.5 * log(sigma2 * (sigma2 + nP * v) / ((sigma2 + nL * v) * (sigma2 + nR * v)));
  return det + v / (2.0 * sigma2) * (QL + QR - QP);
}

/* Conditional posterior of a leaf with n points and partial-residual sum S
 * (sec. 3.3 items 4 and 10): precision n/sigma^2 + 1/sigma_mu^2. */
void oc_leaf_posterior(double n, double S, double sigma2, double mu_mu, double sigma_mu,
                       double *mean, double *prec) {
  double v = sigma_mu * sigma_mu;
  *prec = n / sigma2 + 1.0 / v;
  *mean = (S / sigma2 + mu_mu / v) / *prec;
}

/* Data-independent part of log r for the move on tree (axis, cut);
 * *scale accumulates |terms|.  GROW turns leaf eta of T into a node with
 * rule (a, s) giving T'; PRUNE removes the two leaf children of eta giving
 * T-.  The ratio is prior ratio x reverse/forward proposal probability;
 * the 1/(p_adj * avail) factors of prior and proposal cancel. */
static double log_ratio_prior(const oc_config *c, const int32_t *n_cuts,
                              const uint16_t *axis_in, const uint8_t *cut_in, int32_t move,
                              int32_t eta, int32_t a, int32_t s, double *scale) {
  int32_t H = 1 << (c->D - 1);
  uint16_t *axis = malloc(sizeof(uint16_t) * H);
  uint8_t *big = malloc(H), *small = malloc(H);
  int32_t *G = malloc(sizeof(int32_t) * 2 * H), *P = malloc(sizeof(int32_t) * 2 * H);
  scratch sc = {malloc(sizeof(int32_t) * c->p), malloc(sizeof(int32_t) * c->p)};
  memcpy(axis, axis_in, sizeof(uint16_t) * H);
  memcpy(big, cut_in, H);
  memcpy(small, cut_in, H);
  /* big = tree with eta split, small = tree with eta a leaf */
  if (move == 1) {
    axis[eta] = (uint16_t)a;
    big[eta] = (uint8_t)s;
  } else {
    small[eta] = 0;
  }
  if (2 * eta < H) big[2 * eta] = 0;
  if (2 * eta + 1 < H) big[2 * eta + 1] = 0;
  int32_t nGs, nPs, nGb, nPb;
  move_lists(c, n_cuts, axis, small, G, &nGs, P, &nPs, &sc);
  move_lists(c, n_cuts, axis, big, G, &nGb, P, &nPb, &sc);
  double pg_small = prob_grow(c, nGs, nPs), pg_big = prob_grow(c, nGb, nPb);
  double ps_eta = psplit_of(c, n_cuts, axis, small, eta, &sc);
  double ps_l = psplit_of(c, n_cuts, axis, big, 2 * eta, &sc);
  double ps_r = psplit_of(c, n_cuts, axis, big, 2 * eta + 1, &sc);
  /* log of pi(big)/pi(small) x q(big->small)/q(small->big) */
  double t[8] = {log(ps_eta),  -log(1.0 - ps_eta), log(1.0 - ps_l),        log(1.0 - ps_r),
                 log(1.0 - pg_big), -log((double)nPb), -log(pg_small), log((double)nGs)};
  double lr = 0.0, sc_sum = 0.0;
  for (int k = 0; k < 8; k++) {
    lr += t[k];
    sc_sum += fabs(t[k]);
  }
  if (scale) *scale += sc_sum;
  free(axis);
  free(big);
  free(small);
  free(G);
  free(P);
  free(sc.lo);
  free(sc.hi);
  return move == 1 ? lr : -lr;
}

static int32_t idx_get(const void *row, int bytes, int64_t i) {
  return bytes == 1 ? ((const uint8_t *)row)[i] : ((const uint16_t *)row)[i];
}

static void idx_set(void *row, int bytes, int64_t i, int32_t v) {
  if (bytes == 1)
    ((uint8_t *)row)[i] = (uint8_t)v;
  else
    ((uint16_t *)row)[i] = (uint16_t)v;
}

/* leaf of observation i in the larger tree of the move (sec. 3.3
 * "Traverse indices cache": the cache is updated from the larger tree) */
static int32_t larger_leaf(int32_t move, int32_t eta, int32_t a, int32_t s, const uint8_t *X,
                           int64_t ldx, int64_t i, int32_t c) {
  if (move == 1 && c == eta) return 2 * eta + (X[(int64_t)a * ldx + i] >= s ? 1 : 0);
  return c;
}

/* Value of the current tree at larger-tree leaf h: the two GROW children
 * inherit the value of eta (sec. 3.3 item 8). */
static float old_value(int32_t move, int32_t eta, const float *leaf, int32_t h) {
  if (move == 1 && (h >> 1) == eta) return leaf[eta];
  return leaf[h];
}

/* Data pass (sec. 3.3 items 3 and 7): counts and fp64 residual sums per
 * larger-tree leaf, then partial sums S_h = R_h + n_h * old value (item 8). */
static void leaf_stats(const oc_config *c, const uint8_t *X, int64_t ldx, const float *leaf,
                       const void *idx_row, const float *resid, int32_t move, int32_t eta,
                       int32_t a, int32_t s, int64_t *cnt, double *S) {
  int32_t H = 1 << (c->D - 1);
  for (int32_t h = 0; h < 2 * H; h++) {
    cnt[h] = 0;
    S[h] = 0.0;
  }
  for (int64_t i = 0; i < c->n; i++) {
    int32_t cp = larger_leaf(move, eta, a, s, X, ldx, i, idx_get(idx_row, c->idx_bytes, i));
    cnt[cp] += 1;
    S[cp] += (double)resid[i];
  }
  for (int32_t h = 1; h < 2 * H; h++)
    if (cnt[h] > 0) S[h] += (double)cnt[h] * (double)old_value(move, eta, leaf, h);
}

double oc_log_ratio(const oc_config *c, const int32_t *n_cuts, const uint8_t *X, int64_t ldx,
                    const uint16_t *axis, const uint8_t *cut, const float *leaf,
                    const void *idx_row, const float *resid, double sigma2, int32_t move,
                    int32_t eta, int32_t a, int32_t s, double *scale) {
  int32_t H = 1 << (c->D - 1);
  int64_t *cnt = malloc(sizeof(int64_t) * 2 * H);
  double *S = malloc(sizeof(double) * 2 * H);
  leaf_stats(c, X, ldx, leaf, idx_row, resid, move, eta, a, s, cnt, S);
  if (scale) *scale = 0.0;
  double lr = log_ratio_prior(c, n_cuts, axis, cut, move, eta, a, s, scale);
  double llr = oc_llr(sigma2, c->mu_mu, c->sigma_mu, (double)cnt[2 * eta], S[2 * eta],
                      (double)cnt[2 * eta + 1], S[2 * eta + 1]);
  if (scale) *scale += fabs(llr);
  free(cnt);
  free(S);
  return move == 1 ? lr + llr : lr - llr;
}

/* Leaf of observation i in one heap-stored tree (sec. 3.2: node h has
 * children 2h and 2h+1, nodes of the last level D-1 are always leaves, and a
 * node with cut 0 is a leaf): start at the root and, while the node splits,
 * go right iff the observation's bin on the node's axis reaches the cut.
 * This is the leaf Algorithm 1 computes; the recursive-descent pin checks the
 * two agree. */
int32_t oc_route(int32_t D, const uint16_t *axis, const uint8_t *cut, const uint8_t *X,
                 int64_t ldx, int64_t i) {
  const int32_t first_leaf_level = 1 << (D - 1);
  int32_t h = 1;
  while (h < first_leaf_level && cut[h] != 0) {
    const uint8_t bin = X[(int64_t)axis[h] * ldx + i];
    h = 2 * h + (bin >= cut[h] ? 1 : 0);
  }
  return h;
}

/* ------------------------------------------------------------------ */
/* One step of the sweep (sec. 2.2 "The BART MCMC", sec. 3.3).          */

static void tree_step(const oc_config *c, const int32_t *n_cuts, const uint8_t *X, int64_t ldx,
                      oc_state *st, uint64_t seed, int32_t force, const float *adopt,
                      oc_trace *tr) {
  const int32_t H = 1 << (c->D - 1);
  const int32_t j = st->next;
  const uint64_t s = (uint64_t)st->sweep;
  uint16_t *axis = st->axis + (int64_t)j * H;
  uint8_t *cut = st->cut + (int64_t)j * H;
  float *leaf = st->leaf + (int64_t)j * 2 * H;
  void *idx_row = (char *)st->idx + (int64_t)j * c->n * c->idx_bytes;

  /* 1-2: propose (sec. 3.3 item 1) */
  uint64_t w[4];
  block(seed, (uint32_t)c->chain, s, (uint64_t)j, 0, 0, w);
  int32_t prop[6];
  oc_propose(c, n_cuts, axis, cut, w, prop);
  int32_t move = prop[0], eta = prop[1], a = prop[2], sc = prop[3];
  double ln_u = log(u01(w[3]));

  /* 3-4: counts and partial residual sums of the larger tree */
  int64_t *cnt = malloc(sizeof(int64_t) * 2 * H);
  double *S = malloc(sizeof(double) * 2 * H);
  int32_t *big_leaf = calloc(2 * H, sizeof(int32_t));
  leaf_stats(c, X, ldx, leaf, idx_row, st->resid, move, eta, a, sc, cnt, S);
  for (int32_t h = 1; h < 2 * H; h++) big_leaf[h] = is_leaf_node(cut, H, h);
  if (move == 1) {
    big_leaf[eta] = 0;
    big_leaf[2 * eta] = 1;
    big_leaf[2 * eta + 1] = 1;
  }
  int32_t n_big = 0;
  for (int32_t h = 1; h < 2 * H; h++) n_big += big_leaf[h];

  /* 5: Metropolis-Hastings accept/reject (sec. 3.3 item 9) */
  double log_r = 0.0, scale = 0.0;
  int32_t accept = 0;
  if (move != 0) {
    double lr = log_ratio_prior(c, n_cuts, axis, cut, move, eta, a, sc, &scale);
    double llr = oc_llr(st->sigma2, c->mu_mu, c->sigma_mu, (double)cnt[2 * eta], S[2 * eta],
                        (double)cnt[2 * eta + 1], S[2 * eta + 1]);
    scale += fabs(llr);
    log_r = move == 1 ? lr + llr : lr - llr;
    accept = ln_u < log_r;
    if (force >= 0) accept = force;
  }
  if (tr) {
    memset(tr, 0, sizeof(*tr));
    tr->kind = 0;
    tr->tree = j;
    tr->sweep = st->sweep;
    tr->move = move;
    tr->eta = eta;
    tr->axis = a;
    tr->cut = sc;
    tr->n_grow_cand = prop[4];
    tr->n_prune_cand = prop[5];
    tr->accept = accept;
    tr->n_leaves = n_big;
    tr->log_r = log_r;
    tr->ln_u = ln_u;
    tr->log_r_scale = scale;
    tr->sigma2 = st->sigma2;
    for (int32_t h = 1; h < 2 * H; h++)
      if (big_leaf[h]) {
        tr->count[h] = (int32_t)cnt[h];
        tr->sum[h] = S[h];
      }
  }

  /* 6: final tree; merge the children when the smaller tree is kept */
  float *old = malloc(sizeof(float) * 2 * H);
  memcpy(old, leaf, sizeof(float) * 2 * H);
  int merged = (move == 1 && !accept) || (move == 2 && accept);
  int32_t *fin_leaf = malloc(sizeof(int32_t) * 2 * H);
  memcpy(fin_leaf, big_leaf, sizeof(int32_t) * 2 * H);
  if (move == 1 && accept) {
    axis[eta] = (uint16_t)a;
    cut[eta] = (uint8_t)sc;
    if (2 * eta < H) cut[2 * eta] = 0;
    if (2 * eta + 1 < H) cut[2 * eta + 1] = 0;
  }
  if (move == 2 && accept) cut[eta] = 0;
  if (merged) {
    cnt[eta] = cnt[2 * eta] + cnt[2 * eta + 1];
    S[eta] = S[2 * eta] + S[2 * eta + 1];
    fin_leaf[2 * eta] = 0;
    fin_leaf[2 * eta + 1] = 0;
    fin_leaf[eta] = 1;
  }

  /* 7: draw every leaf of the final tree from its conditional posterior
   * (sec. 2.2; sec. 3.3 items 4, 5 and 10) */
  float *fresh = calloc(2 * H, sizeof(float));
  for (int32_t h = 1; h < 2 * H; h++) {
    if (!fin_leaf[h]) continue;
    double mean, prec;
    oc_leaf_posterior((double)cnt[h], S[h], st->sigma2, c->mu_mu, c->sigma_mu, &mean, &prec);
    double z = normal_of(seed, (uint32_t)c->chain, s, (uint64_t)j, (uint64_t)h);
    fresh[h] = (float)(mean + z / sqrt(prec));
    if (tr) tr->leaf_new[h] = fresh[h];
    /* lockstep hook: carry on from another implementation's draws */
    if (adopt) fresh[h] = adopt[h];
    leaf[h] = fresh[h];
  }

  /* 8: residual cache and index cache (sec. 3.3 items 11, "Residuals cache") */
  for (int64_t i = 0; i < c->n; i++) {
    int32_t ci = idx_get(idx_row, c->idx_bytes, i);
    int32_t cp = larger_leaf(move, eta, a, sc, X, ldx, i, ci);
    int32_t f = (merged && (cp >> 1) == eta) ? eta : cp;
    float delta = old[ci] - fresh[f];
    st->resid[i] = st->resid[i] + delta;
    idx_set(idx_row, c->idx_bytes, i, f);
  }
  free(cnt);
  free(S);
  free(big_leaf);
  free(old);
  free(fin_leaf);
  free(fresh);
}

/* Probit: new latents given the trees, f_i = z_i - r_i (offset included),
 * one uniform per observation from block (s, 2^64 - 2, 3, c 2^32 + i/4),
 * word i mod 4.  The latent is stored in f32 on its side of 0 and the
 * residual follows it: r_i = z_i - f_i. */
static void latent_step(const oc_config *c, oc_state *st, uint64_t seed) {
  uint64_t w[4];
  for (int64_t i = 0; i < c->n; i++) {
    if ((i & 3) == 0) block(seed, (uint32_t)c->chain, (uint64_t)st->sweep, ~1ULL, 3, (uint64_t)(i >> 2), w);
    double u = u01(w[i & 3]);
    double f = (double)st->latent[i] - (double)st->resid[i];
    int y = st->ybin[i] != 0;
    float z = (float)oc_latent_draw(f, y, u);
    if (y && !(z > 0.0f)) z = FLT_MIN;
    if (!y && z > 0.0f) z = 0.0f;
    st->latent[i] = z;
    st->resid[i] = (float)((double)z - f);
  }
}

static void sigma_step(const oc_config *c, oc_state *st, uint64_t seed, oc_trace *tr) {
  double ssr = 0.0;
  for (int64_t i = 0; i < c->n; i++) ssr += (double)st->resid[i] * (double)st->resid[i];
  if (c->probit)
    latent_step(c, st, seed);
  else if (!c->fix_sigma2)
    st->sigma2 = sigma2_of(seed, (uint32_t)c->chain, (uint64_t)st->sweep, c->nu, c->lambda, c->n,
                           ssr);
  if (tr) {
    memset(tr, 0, sizeof(*tr));
    tr->kind = 1;
    tr->tree = c->m;
    tr->sweep = st->sweep;
    tr->ssr = ssr;
    tr->sigma2 = st->sigma2;
  }
}

int oc_step(const oc_config *c, const int32_t *n_cuts, const uint8_t *X, int64_t ldx,
            oc_state *st, uint64_t seed, int32_t force, const float *adopt, oc_trace *trace) {
  if (c->D < 2 || c->D > 8 || c->chain < 0 || st->next < 0 || st->next > c->m) return -1;
  if (st->next < c->m) {
    tree_step(c, n_cuts, X, ldx, st, seed, force, adopt, trace);
    st->next += 1;
  } else {
    sigma_step(c, st, seed, trace);
    st->next = 0;
    st->sweep += 1;
  }
  return 0;
}

int oc_run(const oc_config *c, const int32_t *n_cuts, const uint8_t *X, int64_t ldx,
           oc_state *st, uint64_t seed, int64_t n_steps, oc_trace *traces) {
  for (int64_t k = 0; k < n_steps; k++) {
    int rc = oc_step(c, n_cuts, X, ldx, st, seed, -1, NULL, traces ? traces + k : NULL);
    if (rc) return rc;
  }
  return 0;
}

/* f(x) = offset + sum_j g(x; T_j, M_j) (eq. bartdef), each tree by
 * Algorithm 1, summed in fp64 in tree order. */
void oc_predict(const oc_config *c, const uint16_t *axis, const uint8_t *cut, const float *leaf,
                const uint8_t *Xt, int64_t ldxt, int64_t nt, double offset, float *out) {
  int32_t H = 1 << (c->D - 1);
  for (int64_t i = 0; i < nt; i++) {
    double acc = 0.0;
    for (int32_t j = 0; j < c->m; j++) {
      int32_t h = oc_route(c->D, axis + (int64_t)j * H, cut + (int64_t)j * H, Xt, ldxt, i);
      acc += (double)leaf[(int64_t)j * 2 * H + h];
    }
    out[i] = (float)(offset + acc);
  }
}
