"""Predictive accuracy on the paper's simulated data (sec. 4.2, eq. rmsedgp)
and prediction at scale.

The data have unit noise variance and a signal of variance about 2, so a
sampler that works predicts the test responses with an RMSE near 1 and the
noiseless function with an RMSE well below the signal sd (about 1.4); the
oracle is checked on the CPU, the device path through libbart."""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle
from paper_2410_23244_amd.inputs import bin_column, cutpoints, default_hyper, rmse_dgp


def _oracle_fit(n_train, p=10, m=200, burn=200, keep=200, seed=0):
    Xtr, ytr, Xte, yte, fte = rmse_dgp(n_train, 1000, p, seed)
    K = 255
    cuts = [cutpoints(Xtr[a], K, "quantile") for a in range(p)]
    Xb = np.stack([bin_column(Xtr[a], cuts[a]) for a in range(p)])
    Xtb = np.stack([bin_column(Xte[a], cuts[a]) for a in range(p)])
    off = float(ytr.mean())
    h = default_hyper(ytr - off, m)
    cfg = oracle.make_config(n=n_train, p=p, m=m, D=6, alpha=h.alpha, beta=h.beta, mu_mu=0.0,
                             sigma_mu=h.sigma_mu, nu=h.nu, lam=h.lam)
    ch = oracle.Chain(cfg, Xb, np.full(p, K, np.int32), (ytr - off).astype(np.float32),
                      h.sigma2_init)
    ch.sweeps(seed + 1, burn)
    acc = np.zeros(Xte.shape[1])
    for _ in range(keep):
        ch.sweeps(seed + 1, 1)
        acc += ch.predict(Xtb, off)
    fhat = acc / keep
    return (math.sqrt(np.mean((fhat - yte) ** 2)), math.sqrt(np.mean((fhat - fte) ** 2)),
            math.sqrt(ch.sigma2), float(np.std(fte)))


def test_oracle_rmse_on_the_paper_dgp():
    ry5, rf5, s5, sf = _oracle_fit(500)
    ry2, rf2, s2, _ = _oracle_fit(2000)
    assert sf > 1.2                          # the signal is there to be learnt
    assert rf5 < 0.6 and rf2 < 0.45, (rf5, rf2)
    assert rf2 < rf5                         # more data, better fit
    assert abs(ry2 - 1.0) < 0.15, ry2        # test RMSE near the noise sd
    assert 0.8 < s2 < 1.2, s2                # and so is the sigma draw


@pytest.mark.gpu
def test_device_rmse_on_the_paper_dgp():
    from paper_2410_23244_amd.bart import Regressor

    Xtr, ytr, Xte, yte, fte = rmse_dgp(2000, 1000, 10, 0)
    r = Regressor(ntree=200, nchain=2, seed=5).fit(Xtr.T, ytr, Xte.T, n_burn=200, n_keep=300)
    rmse_y = math.sqrt(np.mean((r.mean - yte) ** 2))
    rmse_f = math.sqrt(np.mean((r.mean - fte) ** 2))
    print(f"device: rmse_y {rmse_y:.3f} rmse_f {rmse_f:.3f} "
          f"sigma {math.sqrt(r.sigma2_trace[-50:].mean()):.3f}", flush=True)
    assert rmse_f < 0.45 and abs(rmse_y - 1.0) < 0.15, (rmse_y, rmse_f)
    assert 0.8 < math.sqrt(r.sigma2_trace[-50:].mean()) < 1.2
    # the chains agree with each other to well within the signal sd (their
    # posterior means carry Monte Carlo error of the order of rmse_f)
    chain_mean = r.sums[0] / r.n_keep
    assert math.sqrt(np.mean((chain_mean[0] - chain_mean[1]) ** 2)) < 0.4
    # posterior sd of f: positive, below the prior scale
    assert (r.sd > 0).all() and np.median(r.sd) < 0.6
    # the oracle on the same data lands at the same accuracy
    ry, rf, _, _ = _oracle_fit(2000)
    assert abs(rmse_f - rf) < 0.1 and abs(rmse_y - ry) < 0.05


@pytest.mark.gpu
def test_predict_at_scale_matches_oracle():
    from paper_2410_23244_amd.bart import from_inputs
    from paper_2410_23244_amd.inputs import make_inputs
    from tests import parity

    inp = make_inputs(5, n=20011, p=1000, m=120)      # depth 8, 1000 predictors
    g = from_inputs(inp, nchain=2)
    g.step(6, 9)
    Xt = make_inputs(5, n=60013, p=1000, m=120).X_b
    got = g.predict(Xt, inp.offset).cpu().numpy()
    for c in range(2):
        ch = parity.chain_from_state(inp, g.get_state(c), chain=c)
        np.testing.assert_array_equal(got[c], ch.predict(Xt, inp.offset))


@pytest.mark.gpu
def test_predict_accumulate_sums_the_kept_sweeps():
    import torch

    from paper_2410_23244_amd.bart import from_inputs
    from paper_2410_23244_amd.inputs import make_inputs

    inp = make_inputs(2, n=5003, p=20, m=40)
    g = from_inputs(inp, nchain=3)
    Xt = make_inputs(2, n=777, p=20, m=40).X_b
    Xd, nt = g.upload_x(Xt)
    s = torch.zeros((3, nt), dtype=torch.float64, device=g.device)
    s2 = torch.zeros_like(s)
    want = np.zeros((3, nt))
    want2 = np.zeros((3, nt))
    g.step(2, 4)
    for _ in range(5):
        g.step(1, 4)
        g.predict_accumulate(Xd, nt, inp.offset, s, s2)
        f = g.predict(Xt, inp.offset).cpu().numpy().astype(np.float64)  # fp32-rounded f
        want += f
        want2 += f * f
    got, got2 = s.cpu().numpy(), s2.cpu().numpy()
    # the accumulator adds f before its rounding to fp32
    tol = 5 * 6e-8 * np.abs(want).max()
    assert np.abs(got - want).max() <= tol
    assert np.abs(got2 - want2).max() <= 2 * tol * np.abs(want).max()
    # pooled posterior mean and sd over the 3 chains (law of total variance)
    mean, sd = g.posterior_summary(s, s2, nt, 5)
    m_c = got / 5
    v_c = got2 / 5 - m_c ** 2
    np.testing.assert_allclose(mean.cpu().numpy(), m_c.mean(axis=0), rtol=1e-12, atol=1e-12)
    want_sd = np.sqrt(np.maximum(v_c.mean(axis=0) + m_c.var(axis=0), 0.0))
    np.testing.assert_allclose(sd.cpu().numpy(), want_sd, rtol=1e-9, atol=1e-9)
    assert g.status() == 0
