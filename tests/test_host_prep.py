"""Host-side input preparation of libbart (no GPU): splitting grids, binning
and default hyperparameters against their definitions (sec. 2.1
"Hyperparameters", sec. 3.2 "Predictors") as numpy and scipy compute them."""
from __future__ import annotations

import ctypes as C
import math
import os

import numpy as np
import pytest
from scipy import stats


@pytest.fixture(scope="module")
def b():
    from paper_2410_23244_amd import bart

    if not os.path.exists(bart.LIB_PATH):
        pytest.skip("libbart.so not built")
    return bart


def _numpy_cuts(x, K, grid):
    x = np.asarray(x, np.float64)
    if grid == 0:
        lo, hi = x.min(), x.max()
        return lo + np.arange(1, K + 1, dtype=np.float64) * (hi - lo) / (K + 1)
    return np.quantile(x, np.arange(1, K + 1, dtype=np.float64) / (K + 1))


@pytest.mark.parametrize("grid,K,n", [(0, 100, 3001), (1, 255, 5000), (1, 17, 40), (0, 255, 7)])
def test_grid_and_bins_match_their_definition(b, grid, K, n):
    rng = np.random.default_rng([7, grid, K, n])
    p = 6
    X = (rng.standard_normal((p, n)) * rng.uniform(0.1, 10, (p, 1))).astype(np.float32)
    cuts, nc = b.bart_cutpoints(X, K, grid)
    Xb = b.bart_bin(X, cuts, nc)
    for a in range(p):
        want = _numpy_cuts(X[a], K, grid)
        want = want[want > X[a].min()] if grid == 1 else want
        want = np.unique(want)
        assert nc[a] == want.size
        np.testing.assert_allclose(cuts[a, : nc[a]], want, rtol=1e-15, atol=0)
        assert np.all(np.isinf(cuts[a, nc[a]:]))
        # x_b = #{k : c_k <= x}, from the library's own cuts
        ref = np.searchsorted(cuts[a, : nc[a]], X[a].astype(np.float64), side="right")
        np.testing.assert_array_equal(Xb[a], ref)
        # and from numpy's: identical for data without ties at a cut
        ref2 = np.searchsorted(want, X[a].astype(np.float64), side="right")
        np.testing.assert_array_equal(Xb[a], ref2)


def test_degenerate_predictors(b):
    n = 1000
    X = np.zeros((3, n), np.float32)
    X[1] = np.arange(n) % 2            # binary: one useful cut
    X[2] = np.arange(n) % 5            # five levels
    for grid in (0, 1):
        cuts, nc = b.bart_cutpoints(X, 255, grid)
        Xb = b.bart_bin(X, cuts, nc)
        assert nc[0] == 0 and (Xb[0] == 0).all()
        # every level of a discrete predictor lands in its own bin
        assert len(np.unique(Xb[1])) == 2 and len(np.unique(Xb[2])) == 5
        for a in range(3):
            assert np.all(np.diff(cuts[a, : nc[a]]) > 0)
    # NaN bins to 0
    Xn = np.array([[0.1, np.nan, 0.7, 0.3]], np.float32)
    cuts = np.array([[0.2, 0.5]], np.float64)
    np.testing.assert_array_equal(b.bart_bin(Xn, cuts, np.array([2], np.int32))[0], [0, 0, 2, 1])


def test_default_hyperparameters(b):
    from paper_2410_23244_amd.inputs import default_hyper

    rng = np.random.default_rng(3)
    for n, m in [(1000, 200), (37, 50), (20000, 1)]:
        y = rng.standard_normal(n) * 3.0 + 5.0
        off, yc, cfg = b.bart_default_hyper(y, m)
        assert off == pytest.approx(y.mean(), rel=1e-14)
        np.testing.assert_array_equal(yc, (y - y.mean()).astype(np.float32))
        h = default_hyper(y - y.mean(), m)
        assert cfg.sigma_mu == pytest.approx(h.sigma_mu, rel=1e-12)
        assert cfg.lam == pytest.approx(h.lam, rel=1e-10)
        assert cfg.sigma2_init == pytest.approx(h.sigma2_init, rel=1e-12)
        assert (cfg.alpha, cfg.beta, cfg.mu_mu, cfg.nu, cfg.p_grow) == (0.95, 2.0, 0.0, 3.0, 0.5)
    # the chi-square quantile behind lambda, at several degrees of freedom
    # through var(y) = 1: lambda = q_0.1(chi2_nu) / nu with nu = 3
    y = np.array([-1.0, 1.0])
    _, _, cfg = b.bart_default_hyper(y, 1)
    assert cfg.lam == pytest.approx(stats.chi2.ppf(0.1, 3) / 3, rel=1e-12)


def test_prep_rejects_invalid_arguments(b):
    L = b.lib()
    X = np.ones((2, 10), np.float32)
    cuts = np.zeros((2, 4))
    nc = np.zeros(2, np.int32)
    assert L.bart_cutpoints(X.ctypes.data, 10, 2, 10, 0, 1, cuts.ctypes.data, nc.ctypes.data) == b.BART_EINVAL
    assert L.bart_cutpoints(X.ctypes.data, 10, 2, 10, 4, 7, cuts.ctypes.data, nc.ctypes.data) == b.BART_EINVAL
    assert L.bart_cutpoints(X.ctypes.data, 10, 2, 5, 4, 1, cuts.ctypes.data, nc.ctypes.data) == b.BART_EINVAL
    Xn = X.copy()
    Xn[1, 3] = np.inf
    assert L.bart_cutpoints(Xn.ctypes.data, 10, 2, 10, 4, 1, cuts.ctypes.data, nc.ctypes.data) == b.BART_EINVAL
    bad = np.array([[1.0, 0.5, 2.0, 3.0], [0, 0, 0, 0]])
    out = np.zeros((2, 10), np.uint8)
    assert L.bart_bin(X.ctypes.data, 10, 2, 10, bad.ctypes.data, np.array([3, 0], np.int32).ctypes.data,
                      4, out.ctypes.data, 10) == b.BART_EINVAL
    y = np.array([1.0, np.nan])
    yc = np.zeros(2, np.float32)
    off = C.c_double()
    cfg = b.Config()
    assert L.bart_default_hyper(y.ctypes.data, 2, 10, C.byref(off), yc.ctypes.data, C.byref(cfg)) == b.BART_EINVAL
