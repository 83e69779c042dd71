"""Seeded synthetic inputs for the BART sweep: predictors, binning, response and
prior hyperparameters.

This module holds no part of the MCMC arithmetic.  It produces the binned
predictor matrix, the centred response and the hyperparameters that both the
HIP path and the CPU oracle take as inputs, so the two sides start from
identical data.

* Predictors are replaced by their index in the splitting grid, 1 byte each
  (sec. 3.2 "Predictors"): ``x_b = #{k : c_k <= x}`` in ``[0, K_a]``, so that
  "go right iff ``x_b >= s``" means ``x >= c_s`` (Algorithm 1).
* Grids (sec. 2.1 "Hyperparameters"): ``K`` evenly spaced cuts strictly inside
  the data range, or ``K`` empirical quantiles.
* Hyperparameter defaults (sec. 2.1): ``mu_mu = 0`` for centred data, ``sigma_mu``
  from the data range, ``nu = 3``, ``lambda`` from the data variance.  The paper
  only says "some measure of location and scale"; the readings used here are
  listed with the design notes.

Each predictor column is drawn from its own counter-seeded numpy generator
(``default_rng([2410, 23244, config, column])``), so columns can be generated
and binned one at a time and the 10^7-row workload never holds its fp32
matrix whole.
"""
from __future__ import annotations

import math
import os
from dataclasses import dataclass, field

import numpy as np

SEED_BASE = (2410, 23244)

# The five synthetic workloads: (n, p, n_tree, depth D, sweeps, cut grid,
# number of cuts, response generator, noise sd, index-cache bytes).
WORKLOADS = {
    1: dict(n=1_000, p=10, m=50, D=6, sweeps=100, grid="uniform", K=100, gen="sin5",
            noise=0.5, idx_bytes=1),
    2: dict(n=100_000, p=100, m=200, D=6, sweeps=1000, grid="quantile", K=255, gen="sin10x",
            noise=1.0, idx_bytes=1),
    3: dict(n=1_000_000, p=100, m=200, D=6, sweeps=1000, grid="quantile", K=255,
            gen="sin10x", noise=1.0, idx_bytes=1),
    4: dict(n=10_000_000, p=100, m=200, D=6, sweeps=200, grid="quantile", K=255,
            gen="sin10x", noise=1.0, idx_bytes=2),
    5: dict(n=1_000_000, p=1000, m=1000, D=8, sweeps=200, grid="quantile", K=255,
            gen="sin10x", noise=1.0, idx_bytes=1),
}


@dataclass
class Hyper:
    alpha: float = 0.95
    beta: float = 2.0
    mu_mu: float = 0.0
    sigma_mu: float = 1.0
    nu: float = 3.0
    lam: float = 1.0
    sigma2_init: float = 1.0
    p_grow: float = 0.5


@dataclass
class Inputs:
    config: int
    n: int
    p: int
    m: int
    D: int
    idx_bytes: int
    sweeps: int
    X_b: np.ndarray            # uint8 [p][n]
    n_cuts: np.ndarray         # int32 [p]
    y_c: np.ndarray            # float32 [n], centred response
    offset: float              # mean of y (fp64), added back by predict
    hyper: Hyper = field(default_factory=Hyper)
    seed: int = 0
    probit: bool = False       # y_c holds binary y (0/1); offset is the probit offset

    @property
    def workload(self) -> str:
        return (f"bart_sweep_n{self.n}_p{self.p}_ntree{self.m}_D{self.D}"
                f"_idx{8 * self.idx_bytes}")


def column(config: int, a: int, n: int) -> np.ndarray:
    """Predictor column a, U[0,1) in fp32."""
    return np.random.default_rng([*SEED_BASE, config, a]).random(n, dtype=np.float32)


def cutpoints(x: np.ndarray, K: int, grid: str) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    if grid == "uniform":
        lo, hi = float(x.min()), float(x.max())
        return lo + np.arange(1, K + 1, dtype=np.float64) * (hi - lo) / (K + 1)
    if grid == "quantile":
        return np.quantile(x, np.arange(1, K + 1, dtype=np.float64) / (K + 1))
    raise ValueError(grid)


def bin_column(x: np.ndarray, cuts: np.ndarray) -> np.ndarray:
    """x_b = #{k : c_k <= x}."""
    xb = np.searchsorted(cuts, np.asarray(x, dtype=np.float64), side="right")
    assert xb.max(initial=0) <= 255
    return xb.astype(np.uint8)


def _response(gen: str, cols: dict, n: int) -> np.ndarray:
    if gen == "sin5":
        return sum(np.sin(2.0 * np.pi * cols[j].astype(np.float64)) for j in range(5))
    if gen == "sin10x":
        f = sum(np.sin(2.0 * np.pi * cols[j].astype(np.float64)) for j in range(10))
        return f + 0.5 * cols[10].astype(np.float64) * cols[11].astype(np.float64)
    raise ValueError(gen)


def default_hyper(y: np.ndarray, m: int, nu: float = 3.0, alpha: float = 0.95,
                  beta: float = 2.0) -> Hyper:
    """Defaults for centred y: sigma_mu puts the range of y at +-2 prior sd of
    the sum of m leaves; lambda puts the data variance at the 0.9 quantile of
    the sigma^2 prior; sigma^2 starts at the data variance."""
    from scipy.stats import chi2

    y = np.asarray(y, dtype=np.float64)
    s2 = float(np.var(y))
    rng = float(y.max() - y.min()) if y.size else 1.0
    sigma_mu = rng / (2.0 * 2.0 * math.sqrt(m)) if rng > 0 else 1.0
    lam = s2 * float(chi2.ppf(0.1, nu)) / nu if s2 > 0 else 1.0
    return Hyper(alpha=alpha, beta=beta, mu_mu=0.0, sigma_mu=sigma_mu, nu=nu, lam=lam,
                 sigma2_init=s2 if s2 > 0 else 1.0)


def make_inputs(config: int, n: int | None = None, p: int | None = None,
                m: int | None = None, D: int | None = None,
                idx_bytes: int | None = None) -> Inputs:
    """Inputs of one workload; n, p, m, D may be overridden to get a smaller
    case of the same generator (the seeds of the columns do not change)."""
    w = dict(WORKLOADS[config])
    n = int(n if n is not None else w["n"])
    p = int(p if p is not None else w["p"])
    m = int(m if m is not None else w["m"])
    D = int(D if D is not None else w["D"])
    idx_bytes = int(idx_bytes if idx_bytes is not None else w["idx_bytes"])
    needed = 5 if w["gen"] == "sin5" else 12
    X_b = np.empty((p, n), np.uint8)
    n_cuts = np.full(p, w["K"], np.int32)
    cols = {}

    def one(a: int) -> None:
        # each column is generated, cut and binned on its own (numpy releases
        # the GIL in the heavy calls, so columns run in parallel threads)
        x = column(config, a, n)
        if a < needed:
            cols[a] = x
        X_b[a] = bin_column(x, cutpoints(x, w["K"], w["grid"]))

    threads = min(16, os.cpu_count() or 1, max(p, 1))
    if threads > 1 and n * p >= 1 << 22:
        from concurrent.futures import ThreadPoolExecutor

        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(one, range(p)))
    else:
        for a in range(p):
            one(a)
    for a in range(p, needed):  # informative columns beyond p (tiny test shapes)
        cols[a] = column(config, a, n)
    f = _response(w["gen"], cols, n)
    noise = np.random.default_rng([*SEED_BASE, config, 10**6]).standard_normal(n) * w["noise"]
    y = f + noise
    offset = float(y.mean()) if n else 0.0
    y_c = (y - offset).astype(np.float32)
    hyper = default_hyper(y - offset, m)
    return Inputs(config=config, n=n, p=p, m=m, D=D, idx_bytes=idx_bytes, sweeps=w["sweeps"],
                  X_b=X_b, n_cuts=n_cuts, y_c=y_c, offset=offset, hyper=hyper, seed=config)


def timing_dgp(n: int, p: int) -> tuple[np.ndarray, np.ndarray]:
    """The paper's own timing data (sec. 4.1, "Data generating process"):
    y_i = cos(2 n pi/32 (i-1)/(n-1)), X_ij = (i + (p+1) j) mod 256 with 1-based
    i, j; X is already an index in a 255-cut grid."""
    i = np.arange(1, n + 1, dtype=np.int64)
    X_b = np.empty((p, n), np.uint8)
    for j in range(1, p + 1):
        X_b[j - 1] = ((i + (p + 1) * j) % 256).astype(np.uint8)
    y = np.cos(2.0 * n * np.pi / 32.0 * (i - 1) / max(n - 1, 1))
    return X_b, y


def rmse_dgp(n_train: int, n_test: int, p: int, seed: int = 0):
    """The paper's predictive-accuracy data (sec. 4.2, eq. rmsedgp): a dense
    linear term and a sparse quadratic term, each standardised to unit
    sample variance over train and test together, plus N(0, 1) noise.
    X ~ U(0,1), beta_j ~ N(0,1), A_jk ~ N(0,1) when the circular distance
    min(|j-k|, p-|j-k|) < 5, else 0.  Returns (X_train [p][n_train] f32,
    y_train, X_test [p][n_test] f32, y_test, f_test) with y and f in fp64."""
    rng = np.random.default_rng([*SEED_BASE, 42, seed])
    n = n_train + n_test
    X = rng.random((n, p))
    beta = rng.standard_normal(p)
    j = np.arange(p)
    dist = np.abs(j[:, None] - j[None, :])
    near = np.minimum(dist, p - dist) < 5
    A = np.where(near, rng.standard_normal((p, p)), 0.0)
    lin = X @ beta
    quad = np.einsum("ij,jk,ik->i", X, A, X)
    f = lin / lin.std() + quad / quad.std()
    y = f + rng.standard_normal(n)
    Xf = X.astype(np.float32).T.copy()
    return (Xf[:, :n_train].copy(), y[:n_train], Xf[:, n_train:].copy(), y[n_train:],
            f[n_train:])


def make_probit_inputs(n: int, p: int, m: int, D: int = 6, K: int = 255, seed: int = 0,
                       idx_bytes: int = 1) -> Inputs:
    """Binary-response workload for the probit model: X ~ U[0,1) columns of
    workload 2's generator, P(y = 1 | x) = Phi(g(x)) with
    g = 1.5 sin(2 pi x_0) + 2 (x_1 - 1/2) + x_2 x_3 - 1/4, K quantile cuts.
    y_c holds y in {0, 1}; offset = Phi^-1(mean y); sigma_mu = 3 / (2 sqrt m)
    puts +-3 (probabilities 0.1 % and 99.9 %) at 2 prior sd of the sum of
    trees; sigma^2 = 1."""
    from scipy.stats import norm

    X_b = np.empty((p, n), np.uint8)
    cols = {}
    for a in range(max(p, 4)):
        x = column(2, a, n)
        if a < 4:
            cols[a] = x.astype(np.float64)
        if a < p:
            X_b[a] = bin_column(x, cutpoints(x, K, "quantile"))
    g = (1.5 * np.sin(2.0 * np.pi * cols[0]) + 2.0 * (cols[1] - 0.5) + cols[2] * cols[3]
         - 0.25)
    u = np.random.default_rng([*SEED_BASE, 77, seed]).random(n)
    y = (u < norm.cdf(g)).astype(np.float32)
    ybar = float(y.mean()) if n else 0.5
    offset = float(norm.ppf(min(max(ybar, 1e-6), 1 - 1e-6)))
    hyper = Hyper(sigma_mu=3.0 / (2.0 * math.sqrt(m)), sigma2_init=1.0)
    inp = Inputs(config=2, n=n, p=p, m=m, D=D, idx_bytes=idx_bytes, sweeps=0, X_b=X_b,
                 n_cuts=np.full(p, K, np.int32), y_c=y, offset=offset, hyper=hyper,
                 seed=seed, probit=True)
    return inp
