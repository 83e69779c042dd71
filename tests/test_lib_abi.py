"""Host-side checks of libbart that need no GPU: the library loads, exports
every entry point include/bart.h declares, and rejects invalid arguments
before touching the device."""
from __future__ import annotations

import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bart.h")


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(bart_[a-z_]+)\s*\(", txt)))


@pytest.fixture(scope="module")
def b():
    from paper_2410_23244_amd import bart

    if not os.path.exists(bart.LIB_PATH):
        pytest.skip("libbart.so not built")
    return bart


def test_exports_every_declared_symbol(b):
    names = _declared()
    assert "bart_init" in names and "bart_step" in names and "bart_predict" in names
    L = b.lib()
    missing = [n for n in names if not hasattr(L, n)]
    assert not missing, missing


def _cfg(b, **kw):
    base = dict(n=1000, p=4, ntree=10, max_depth=6, idx_bytes=1, grid=0, launch=0,
                residency=0, nchain=1, probit=0, x_stride=1024,
                alpha=0.95, beta=2.0, mu_mu=0.0, sigma_mu=0.1, nu=3.0, lam=0.5,
                sigma2_init=1.0, p_grow=0.5, probit_offset=0.0)
    base.update(kw)
    return b.Config(*[base[f] for f, _ in b.Config._fields_])


@pytest.mark.parametrize("bad", [dict(n=0), dict(max_depth=1), dict(max_depth=9),
                                 dict(idx_bytes=3), dict(x_stride=1000), dict(x_stride=512),
                                 dict(alpha=1.5), dict(sigma_mu=0.0), dict(nu=-1.0),
                                 dict(p_grow=2.0), dict(grid=300), dict(grid=-1), dict(lam=float("nan")),
                                 dict(launch=2), dict(launch=-1), dict(residency=3),
                                 dict(residency=-1), dict(nchain=-1), dict(nchain=257),
                                 dict(nchain=3, grid=100), dict(probit=2),
                                 dict(probit=1, probit_offset=float("inf"))])
def test_invalid_configs_are_rejected(b, bad):
    cfg = _cfg(b, **bad)
    assert b.bart_workspace_bytes(cfg) == 0
    h = C.c_void_p()
    nc = np.full(4, 10, np.int32)
    rc = b.lib().bart_init(C.byref(cfg), 4096, 4096, nc.ctypes.data, 4096, 1 << 30, None,
                           C.byref(h))
    assert rc == b.BART_EINVAL and h.value is None
    assert b.lib().bart_last_error().decode()


def test_workspace_size_and_alignment_checks(b):
    cfg = _cfg(b)
    need = b.bart_workspace_bytes(cfg)
    # residuals, u8 cache, trees, proposals, normals, mailboxes
    assert need >= 1000 * 4 + 10 * 1024 + 10 * 32 * 3 + 10 * 64 * 8
    h = C.c_void_p()
    nc = np.full(4, 10, np.int32)
    L = b.lib()
    assert L.bart_init(C.byref(cfg), 4096, 4096, nc.ctypes.data, 4096, need - 1, None,
                       C.byref(h)) == b.BART_ENOSPACE
    assert L.bart_init(C.byref(cfg), 4096, 4096, nc.ctypes.data, 4096 + 8, need, None,
                       C.byref(h)) == b.BART_ENOSPACE
    bad = np.array([10, 256, 3, 0], np.int32)
    assert L.bart_init(C.byref(cfg), 4096, 4096, bad.ctypes.data, 4096, need, None,
                       C.byref(h)) == b.BART_EINVAL
    assert L.bart_init(C.byref(cfg), 0, 4096, nc.ctypes.data, 4096, need, None,
                       C.byref(h)) == b.BART_EINVAL


def test_workspace_grows_with_chains(b):
    one = b.bart_workspace_bytes(_cfg(b, nchain=1))
    assert b.bart_workspace_bytes(_cfg(b, nchain=0)) == one  # 0 means one chain
    four = b.bart_workspace_bytes(_cfg(b, nchain=4))
    # every chain has its own residuals, index cache and trees
    assert four >= 4 * (1000 * 4 + 10 * 1024 + 10 * 32 * 3)
    assert four > one


def test_null_handle_calls_fail_cleanly(b):
    L = b.lib()
    assert L.bart_step(None, 1, 0) == b.BART_EINVAL
    assert L.bart_debug_steps(None, 1, 0, None) == b.BART_EINVAL
    assert L.bart_predict(None, None, 16, 1, 0.0, None) == b.BART_EINVAL
    assert L.bart_status(None, None) == b.BART_EINVAL
    L.bart_destroy(None)
