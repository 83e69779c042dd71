"""Values the paper prints (tests/golden/paper_values.txt, each line with its
section) against the library's host interface, the oracle's configuration
defaults and the synthetic workload table.  No GPU."""
from __future__ import annotations

import inspect
import os
from pathlib import Path

import numpy as np
import pytest

GOLDEN = Path(__file__).parent / "golden" / "paper_values.txt"


def _values() -> dict[str, float]:
    out = {}
    for line in GOLDEN.read_text().splitlines():
        if line.strip() and not line.startswith("#"):
            name, value = line.split()[:2]
            out[name] = float(value)
    return out


V = _values()


@pytest.fixture(scope="module")
def b():
    from paper_2410_23244_amd import bart

    if not os.path.exists(bart.LIB_PATH):
        pytest.skip("libbart.so not built")
    return bart


def _cfg(b, **kw):
    base = dict(n=1024, p=4, ntree=10, max_depth=6, idx_bytes=1, grid=0, launch=0,
                residency=0, nchain=1, probit=0, x_stride=1024,
                alpha=0.95, beta=2.0, mu_mu=0.0, sigma_mu=0.1, nu=3.0, lam=0.5,
                sigma2_init=1.0, p_grow=0.5, probit_offset=0.0)
    base.update(kw)
    return b.Config(*[base[f] for f, _ in b.Config._fields_])


def test_fixture_is_complete():
    assert set(V) == {"ntree_default", "alpha_default", "beta_default", "nu_default",
                      "max_cutpoints", "package_cutpoints", "predictor_bytes",
                      "index_max_depth", "index_bytes", "bench_low_p", "bench_low_ntree"}


def test_hyperparameter_defaults(b):
    import oracle
    from paper_2410_23244_amd.inputs import default_hyper

    y = np.random.default_rng(0).standard_normal(500)
    _, _, cfg = b.bart_default_hyper(y, int(V["ntree_default"]))
    assert (cfg.alpha, cfg.beta, cfg.nu) == (V["alpha_default"], V["beta_default"], V["nu_default"])
    h = default_hyper(y - y.mean(), int(V["ntree_default"]))
    assert (h.alpha, h.beta, h.nu) == (V["alpha_default"], V["beta_default"], V["nu_default"])
    d = inspect.signature(oracle.make_config).parameters
    assert (d["alpha"].default, d["beta"].default, d["nu"].default) == (
        V["alpha_default"], V["beta_default"], V["nu_default"])


def test_cutpoint_grid_fits_a_byte(b):
    K = int(V["max_cutpoints"])
    x = np.random.default_rng(1).random((2, 4000)).astype(np.float32)
    cuts, n_cuts = b.bart_cutpoints(x, K, 1)
    assert (n_cuts <= K).all() and n_cuts.max() == K
    xb = b.bart_bin(x, cuts, n_cuts)
    assert xb.dtype.itemsize == V["predictor_bytes"] and xb.max() == K
    with pytest.raises(b.BartError):
        b.bart_cutpoints(x, K + 1, 1)
    # the package default fits too
    cuts, n_cuts = b.bart_cutpoints(x, int(V["package_cutpoints"]), 0)
    assert (n_cuts == V["package_cutpoints"]).all()


def test_index_cache_is_n_ntree_bytes(b):
    n, m = 1024, 10  # n a multiple of the 256-point padding
    one = b.bart_workspace_bytes(_cfg(b, n=n, ntree=m, idx_bytes=1))
    two = b.bart_workspace_bytes(_cfg(b, n=n, ntree=m, idx_bytes=2))
    assert two - one == n * m * V["index_bytes"]
    # one byte holds every heap index up to the paper's depth limit, no further
    D = int(V["index_max_depth"])
    assert b.bart_workspace_bytes(_cfg(b, max_depth=D)) > 0
    assert b.bart_workspace_bytes(_cfg(b, max_depth=D + 1)) == 0


def test_benchmark_workloads_use_the_low_settings():
    from paper_2410_23244_amd.inputs import WORKLOADS

    for c in (2, 3, 4):
        assert (WORKLOADS[c]["p"], WORKLOADS[c]["m"]) == (V["bench_low_p"], V["bench_low_ntree"])
        assert WORKLOADS[c]["K"] == V["max_cutpoints"]
    assert WORKLOADS[1]["K"] == V["package_cutpoints"]
