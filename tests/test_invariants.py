"""The state invariants the GPU tests check after untraced runs, exercised on
oracle chains (no GPU): they hold for a correct state and each catches a
planted mistake."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2410_23244_amd.inputs import make_inputs
from tests import parity


@pytest.fixture(scope="module")
def state():
    inp = make_inputs(1, n=3001, p=10, m=20)
    ch = oracle.Chain(oracle.config_for(inp), inp.X_b, inp.n_cuts, inp.y_c,
                      inp.hyper.sigma2_init)
    ch.sweeps(3, 8)
    H = 1 << (inp.D - 1)
    cnt = np.zeros((inp.m, 2 * H), np.int32)
    for j in range(inp.m):
        cnt[j] = np.bincount(ch.idx[j], minlength=2 * H)[: 2 * H]
    st = dict(axis=ch.axis.copy(), cut=ch.cut.copy(), leaf=ch.leaf.copy(), idx=ch.idx.copy(),
              resid=ch.resid.copy(), count=cnt)
    # at least one tree with a split, so a point can be moved to another leaf
    assert (st["cut"][:, 1] != 0).any()
    return inp, st


def test_holds_for_the_oracle_chain(state):
    inp, st = state
    out = parity.check_invariants(inp, st, sweeps=8, n_sample=inp.n)
    assert out["resid_drift"] <= out["bound"]


def _split_tree(st):
    return int(np.flatnonzero(st["cut"][:, 1] != 0)[0])


def test_catches_a_misrouted_point(state):
    inp, st = state
    bad = {k: v.copy() for k, v in st.items()}
    j = _split_tree(st)
    h = int(bad["idx"][j, 5])
    bad["idx"][j, 5] = h ^ 1  # the sibling slot
    with pytest.raises(AssertionError):
        parity.check_invariants(inp, bad, sweeps=8, n_sample=inp.n)


def test_catches_a_wrong_count(state):
    inp, st = state
    bad = {k: v.copy() for k, v in st.items()}
    j = _split_tree(st)
    bad["count"][j, int(st["idx"][j, 0])] += 1
    with pytest.raises(AssertionError):
        parity.check_invariants(inp, bad, sweeps=8)


def test_catches_residual_drift(state):
    inp, st = state
    bad = {k: v.copy() for k, v in st.items()}
    bad["resid"][7] += 1e-3
    with pytest.raises(AssertionError):
        parity.check_invariants(inp, bad, sweeps=8)
