// prep.hpp -- host-side preparation of BART inputs (part of bart.hip):
// splitting grids, binned predictors and default hyperparameters.  The
// paper moves this work to the CPU and hands the GPU MCMC-ready matrices
// (sec. 4.1, "Caveats about practical performance").
#pragma once

#include <algorithm>
#include <cmath>
#include <thread>
#include <vector>

namespace bart_prep {

// Regularized lower incomplete gamma P(a, x) = gamma(a, x) / Gamma(a), a > 0,
// x >= 0: the power series x^a e^-x / Gamma(a+1) sum_k x^k / ((a+1)...(a+k))
// below x < a + 1, else 1 - Q(a, x) with Q from the Legendre continued
// fraction evaluated by the modified Lentz method.
inline double gamma_p(double a, double x) {
  if (x <= 0.0) return 0.0;
  const double lg = std::lgamma(a);
  if (x < a + 1.0) {
    double term = 1.0 / a, sum = term;
    for (int k = 1; k < 100000; ++k) {
      term *= x / (a + k);
      sum += term;
      if (std::fabs(term) < std::fabs(sum) * 1e-17) break;
    }
    return sum * std::exp(-x + a * std::log(x) - lg);
  }
  const double tiny = 1e-300;
  double b = x + 1.0 - a, c = 1.0 / tiny, d = 1.0 / b, h = d;
  for (int k = 1; k < 100000; ++k) {
    const double an = -k * (k - a);
    b += 2.0;
    d = an * d + b;
    if (std::fabs(d) < tiny) d = tiny;
    c = b + an / c;
    if (std::fabs(c) < tiny) c = tiny;
    d = 1.0 / d;
    const double del = d * c;
    h *= del;
    if (std::fabs(del - 1.0) < 1e-16) break;
  }
  return 1.0 - std::exp(-x + a * std::log(x) - lg) * h;
}

// q-quantile of the chi-square distribution with nu degrees of freedom:
// the root of P(nu/2, x/2) = q, by bisection to fp64 resolution.
inline double chi2_quantile(double q, double nu) {
  double lo = 0.0, hi = std::max(1.0, nu);
  while (gamma_p(0.5 * nu, 0.5 * hi) < q) hi *= 2.0;
  for (int it = 0; it < 200 && hi - lo > 1e-15 * hi; ++it) {
    const double mid = 0.5 * (lo + hi);
    (gamma_p(0.5 * nu, 0.5 * mid) < q ? lo : hi) = mid;
  }
  return 0.5 * (lo + hi);
}

// Linear interpolation between order statistics at probability q (the
// "linear" definition: position q (n - 1) in the sorted sample).
inline double quantile_sorted(const std::vector<double> &v, double q) {
  const size_t n = v.size();
  if (n == 1) return v[0];
  const double pos = q * (double)(n - 1);
  size_t lo = (size_t)std::floor(pos);
  if (lo >= n - 1) return v[n - 1];
  const double t = pos - (double)lo, a = v[lo], b = v[lo + 1];
  return t < 0.5 ? a + (b - a) * t : b - (b - a) * (1.0 - t);
}

// Run f(a) for a in [0, p) on up to 16 host threads.
template <class F>
void for_axes(int p, F f) {
  const int nt = std::max(1, std::min<int>({16, p, (int)std::thread::hardware_concurrency()}));
  if (nt == 1) {
    for (int a = 0; a < p; ++a) f(a);
    return;
  }
  std::vector<std::thread> th;
  for (int k = 0; k < nt; ++k)
    th.emplace_back([&, k] {
      for (int a = k; a < p; a += nt) f(a);
    });
  for (auto &x : th) x.join();
}

}  // namespace bart_prep

extern "C" {

int bart_cutpoints(const float *X, int64_t n, int32_t p, int64_t ldx, int32_t K, int32_t grid,
                   double *cuts, int32_t *n_cuts) {
  if (!X || !cuts || !n_cuts) return fail(BART_EINVAL, "NULL argument");
  if (n < 1 || p < 1 || ldx < n) return fail(BART_EINVAL, "need n >= 1, p >= 1, ldx >= n");
  if (K < 1 || K > 255) return fail(BART_EINVAL, "K must be in [1, 255]");
  if (grid != BART_GRID_UNIFORM && grid != BART_GRID_QUANTILE)
    return fail(BART_EINVAL, "grid must be BART_GRID_UNIFORM or BART_GRID_QUANTILE");
  std::vector<int> bad(p, 0);
  bart_prep::for_axes(p, [&](int a) {
    const float *x = X + (int64_t)a * ldx;
    double *c = cuts + (int64_t)a * K;
    int kept = 0;
    if (grid == BART_GRID_UNIFORM) {
      double lo = INFINITY, hi = -INFINITY;
      for (int64_t i = 0; i < n; ++i) {
        if (!std::isfinite(x[i])) {
          bad[a] = 1;
          return;
        }
        lo = std::min(lo, (double)x[i]);
        hi = std::max(hi, (double)x[i]);
      }
      if (hi > lo)
        for (int k = 1; k <= K; ++k) {
          const double v = lo + ((double)k * (hi - lo)) / (double)(K + 1);
          if (kept == 0 || v > c[kept - 1]) c[kept++] = v;
        }
    } else {
      std::vector<double> v(n);
      for (int64_t i = 0; i < n; ++i) {
        if (!std::isfinite(x[i])) {
          bad[a] = 1;
          return;
        }
        v[i] = x[i];
      }
      std::sort(v.begin(), v.end());
      for (int k = 1; k <= K; ++k) {
        const double q = bart_prep::quantile_sorted(v, (double)k / (double)(K + 1));
        // a cut at or below the minimum separates nothing
        if (q > v[0] && (kept == 0 || q > c[kept - 1])) c[kept++] = q;
      }
    }
    for (int k = kept; k < K; ++k) c[k] = INFINITY;
    n_cuts[a] = kept;
  });
  for (int a = 0; a < p; ++a)
    if (bad[a]) return fail(BART_EINVAL, "X has a non-finite value in predictor %d", a);
  return BART_OK;
}

int bart_bin(const float *X, int64_t n, int32_t p, int64_t ldx, const double *cuts,
             const int32_t *n_cuts, int32_t K, uint8_t *X_b, int64_t ldb) {
  if (!X || !cuts || !n_cuts || !X_b) return fail(BART_EINVAL, "NULL argument");
  if (n < 0 || p < 1 || ldx < n || ldb < n) return fail(BART_EINVAL, "need p >= 1, ldx, ldb >= n");
  if (K < 1 || K > 255) return fail(BART_EINVAL, "K must be in [1, 255]");
  for (int a = 0; a < p; ++a) {
    if (n_cuts[a] < 0 || n_cuts[a] > K) return fail(BART_EINVAL, "n_cuts[%d] not in [0, K]", a);
    const double *c = cuts + (int64_t)a * K;
    for (int k = 1; k < n_cuts[a]; ++k)
      if (!(c[k] > c[k - 1])) return fail(BART_EINVAL, "cuts of predictor %d not increasing", a);
  }
  bart_prep::for_axes(p, [&](int a) {
    const float *x = X + (int64_t)a * ldx;
    const double *c = cuts + (int64_t)a * K;
    const int nc = n_cuts[a];
    uint8_t *o = X_b + (int64_t)a * ldb;
    for (int64_t i = 0; i < n; ++i) {  // #{k : c_k <= x}; NaN goes to 0
      const double v = x[i];
      o[i] = std::isnan(v) ? 0 : (uint8_t)(std::upper_bound(c, c + nc, v) - c);
    }
  });
  return BART_OK;
}

int bart_default_hyper(const double *y, int64_t n, int32_t ntree, double *offset, float *y_c,
                       bart_config *cfg) {
  if (!y || !offset || !y_c || !cfg) return fail(BART_EINVAL, "NULL argument");
  if (n < 1 || ntree < 1) return fail(BART_EINVAL, "need n >= 1 and ntree >= 1");
  double mean = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    if (!std::isfinite(y[i])) return fail(BART_EINVAL, "y[%lld] is not finite", (long long)i);
    mean += y[i];
  }
  mean /= (double)n;
  double ss = 0.0, lo = INFINITY, hi = -INFINITY;
  for (int64_t i = 0; i < n; ++i) {
    const double d = y[i] - mean;
    ss += d * d;
    lo = std::min(lo, d);
    hi = std::max(hi, d);
    y_c[i] = (float)d;
  }
  const double s2 = ss / (double)n;
  const double nu = 3.0;
  *offset = mean;
  cfg->alpha = 0.95;
  cfg->beta = 2.0;
  cfg->mu_mu = 0.0;
  // the range of y at +-2 prior sd of the sum of ntree leaves
  cfg->sigma_mu = hi > lo ? (hi - lo) / (4.0 * std::sqrt((double)ntree)) : 1.0;
  cfg->nu = nu;
  // the data variance at the 0.9 quantile of the sigma^2 prior
  cfg->lambda = s2 > 0.0 ? s2 * bart_prep::chi2_quantile(0.1, nu) / nu : 1.0;
  cfg->sigma2_init = s2 > 0.0 ? s2 : 1.0;
  cfg->p_grow = 0.5;
  return BART_OK;
}

}  // extern "C"
