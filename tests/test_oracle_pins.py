"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: numpy's
Philox, scipy distributions, quadrature, multivariate-normal densities,
exhaustive enumeration of tiny tree spaces, closed forms and the residual
drift bound the paper states (app. B)."""
from __future__ import annotations

import math

import numpy as np
import pytest
from scipy import integrate, stats

import oracle
from tests import treeenum as te

KEY_TAG = 0x42415254


# --------------------------------------------------------------------------
# random numbers

@pytest.mark.parametrize("seed,ctr", [(0, (0, 0, 0, 0)), (123, (5, 7, 1, 3)),
                                      (2**64 - 1, (2**64 - 1, 2**64 - 1, 2, 9)),
                                      (3, (17, 2**63, 1, 31))])
def test_philox_matches_numpy(seed, ctr):
    # numpy increments the 256-bit counter before producing a block
    prev = list(ctr)
    for k in range(4):
        prev[k] = (prev[k] - 1) % 2**64
        if ctr[k] != 0:
            break
    bg = np.random.Philox(key=np.array([seed, KEY_TAG], np.uint64),
                          counter=np.array(prev, np.uint64))
    want = bg.random_raw(4)
    got = oracle.philox(ctr, (seed, KEY_TAG))
    np.testing.assert_array_equal(got, want)


def test_uniform_is_strictly_inside_unit_interval():
    # u_move = u01(w0) with pg = 1 must always choose GROW, even for w0 = 2^64-1
    cfg = oracle.make_config(n=1, p=1, m=1, D=3)
    a0, c0 = te.arrays({}, 3)
    for w0 in [0, 1, 2**64 - 1, 2**64 - 2**11, 2**63]:
        assert oracle.propose(cfg, [4], a0, c0, [w0, 0, 0, 0])[0] == 1


def test_normals_are_standard_normal():
    z = np.array([oracle.normal(11, s, j, h) for s in range(40) for j in range(25)
                  for h in range(2, 22)])
    assert stats.kstest(z, "norm").pvalue > 1e-3
    assert abs(z.mean()) < 4.0 / math.sqrt(z.size)
    assert abs(z.var() - 1.0) < 6.0 * math.sqrt(2.0 / z.size)
    # both normals of one block are used and differ
    assert oracle.normal(1, 2, 3, 4) != oracle.normal(1, 2, 3, 5)


@pytest.mark.parametrize("shape", [2.0, 7.5, 51.5, 5001.5])
def test_gamma_sampler(shape):
    g = np.array([oracle.gamma_draw(7, s, shape) for s in range(6000)])
    assert stats.kstest(g, stats.gamma(shape).cdf).pvalue > 1e-3
    assert abs(g.mean() - shape) < 5.0 * math.sqrt(shape / g.size)


def test_sigma2_draw_is_inverse_gamma():
    nu, lam, n, ssr = 3.0, 0.4, 37, 29.0
    d = np.array([oracle.sigma2_draw(5, s, nu, lam, n, ssr) for s in range(6000)])
    ref = stats.invgamma((nu + n) / 2.0, scale=(nu * lam + ssr) / 2.0)
    assert stats.kstest(d, ref.cdf).pvalue > 1e-3
    mean = (nu * lam + ssr) / (nu + n - 2.0)
    assert abs(d.mean() - mean) < 5.0 * ref.std() / math.sqrt(d.size)


# --------------------------------------------------------------------------
# conjugate pieces

@pytest.mark.parametrize("mu_mu", [0.0, 0.35])
def test_llr_equals_mvn_density_ratio(mu_mu):
    rng = np.random.default_rng(4)
    for trial in range(25):
        nL, nR = int(rng.integers(0, 5)), int(rng.integers(0, 5))
        if nL + nR == 0:
            continue
        sigma2, sigma_mu = float(rng.uniform(0.2, 2)), float(rng.uniform(0.1, 1.5))
        yL, yR = rng.normal(0.5, 1.0, nL), rng.normal(-0.3, 1.0, nR)

        def lm(y):
            if len(y) == 0:
                return 0.0
            cov = sigma2 * np.eye(len(y)) + sigma_mu**2 * np.ones((len(y), len(y)))
            return stats.multivariate_normal(np.full(len(y), mu_mu), cov).logpdf(y)

        want = lm(yL) + lm(yR) - lm(np.concatenate([yL, yR]))
        got = oracle.llr(sigma2, mu_mu, sigma_mu, nL, yL.sum(), nR, yR.sum())
        assert abs(got - want) < 1e-11 * (1 + abs(want)), (trial, got, want)


def test_leaf_posterior_by_quadrature():
    rng = np.random.default_rng(8)
    for n in [0, 1, 3, 40]:
        y = rng.normal(0.7, 1.3, n)
        sigma2, mu_mu, sigma_mu = 0.8, -0.2, 0.6
        mean, prec = oracle.leaf_posterior(n, y.sum(), sigma2, mu_mu, sigma_mu)

        def logd(mu):
            return (stats.norm.logpdf(mu, mu_mu, sigma_mu)
                    + stats.norm.logpdf(y, mu, math.sqrt(sigma2)).sum())

        centre = y.mean() if n else mu_mu
        ref = logd(centre)

        def dens(mu):
            return math.exp(logd(mu) - ref)

        lo, hi = mu_mu - 12 * sigma_mu - 5, mu_mu + 12 * sigma_mu + 5
        pts = [centre, mu_mu]
        Z = integrate.quad(dens, lo, hi, points=pts, limit=400, epsabs=0, epsrel=1e-13)[0]
        m1 = integrate.quad(lambda u: u * dens(u), lo, hi, points=pts, limit=400, epsabs=0,
                            epsrel=1e-13)[0] / Z
        m2 = integrate.quad(lambda u: (u - m1) ** 2 * dens(u), lo, hi, points=pts, limit=400,
                            epsabs=0, epsrel=1e-13)[0] / Z
        assert abs(mean - m1) < 1e-8, (n, mean, m1)
        assert abs(1.0 / prec - m2) < 1e-8, (n, 1 / prec, m2)


# --------------------------------------------------------------------------
# trees: traversal, bookkeeping, prior

def _random_tree(rng, p, n_cuts, D, alpha=0.9, beta=0.5):
    """Draw a tree from the generative prior (test-side, by recursion)."""
    splits = {}
    H = 1 << (D - 1)

    def rec(h, lo, hi):
        d = int(math.floor(math.log2(h)))
        axes = [a for a in range(p) if hi[a] - lo[a] > 0]
        if h >= H or not axes or rng.random() >= alpha * (1 + d) ** (-beta):
            return
        a = axes[rng.integers(len(axes))]
        s = int(rng.integers(lo[a] + 1, hi[a] + 1))
        splits[h] = (a, s)
        hl, lr = list(hi), list(lo)
        hl[a], lr[a] = s - 1, s
        rec(2 * h, lo, hl)
        rec(2 * h + 1, lr, hi)

    rec(1, [0] * p, list(n_cuts))
    return splits


def test_algorithm1_matches_recursive_descent():
    rng = np.random.default_rng(1)
    for D in [2, 3, 6, 8]:
        p, n = 4, 300
        n_cuts = [5, 255, 1, 30]
        X = np.stack([rng.integers(0, k + 1, n) for k in n_cuts]).astype(np.uint8)
        for _ in range(20):
            sp = _random_tree(rng, p, n_cuts, D)
            axis, cut = te.arrays(sp, D)
            # garbage in the ignored entries must not matter
            H = 1 << (D - 1)
            for h in range(1, H):
                if h not in sp:
                    axis[h] = rng.integers(p)
            for i in range(0, n, 7):
                assert oracle.route(D, axis, cut, X, i) == te.descend(sp, X, i)


def test_tree_bookkeeping_against_bruteforce():
    rng = np.random.default_rng(2)
    p, n_cuts, D = 3, [2, 4, 1], 5
    cfg = oracle.make_config(n=1, p=p, m=1, D=D, alpha=0.9, beta=0.7)
    for _ in range(60):
        sp = _random_tree(rng, p, n_cuts, D)
        axis, cut = te.arrays(sp, D)
        info = oracle.tree_info(cfg, n_cuts, axis, cut)
        lv = te.leaves(sp)
        assert sorted(np.nonzero(info["is_leaf"])[0].tolist()) == lv
        assert info["grow"].tolist() == te.growable(sp, p, n_cuts, D, 0.9, 0.7)
        assert info["prune"].tolist() == te.prunable(sp)
        for h in lv:
            lo, hi = te.region(sp, h, p, n_cuts)
            assert info["p_adj"][h] == sum(hi[a] - lo[a] > 0 for a in range(p))


@pytest.mark.parametrize("p,n_cuts,D,alpha,beta", [(1, [3], 3, 0.95, 2.0),
                                                  (2, [2, 1], 3, 0.95, 2.0),
                                                  (2, [3, 2], 3, 0.7, 0.3),
                                                  (2, [2, 2], 4, 0.9, 1.0),
                                                  (1, [0], 4, 0.95, 2.0)])
def test_tree_prior_sums_to_one(p, n_cuts, D, alpha, beta):
    cfg = oracle.make_config(n=1, p=p, m=1, D=D, alpha=alpha, beta=beta)
    total = 0.0
    count = 0
    for sp, lp in te.enumerate_trees(p, n_cuts, D, alpha, beta):
        axis, cut = te.arrays(sp, D)
        lo = oracle.log_prior(cfg, n_cuts, axis, cut)
        assert abs(lo - lp) < 1e-12 or (lo == lp == -math.inf)
        total += math.exp(lo)
        count += 1
    assert abs(total - 1.0) < 1e-12, (total, count)


def test_proposal_is_uniform_over_choices():
    """The pick words map onto the uniform choices of sec. 3.3: every growable
    leaf, available axis and available cut (and every prunable node) is hit by
    a 1/k share of the 32-bit word range."""
    p, n_cuts, D = 3, [3, 0, 5], 4
    cfg = oracle.make_config(n=1, p=p, m=1, D=D, alpha=0.95, beta=2.0, p_grow=0.5)
    sp = {1: (0, 2), 2: (2, 3)}
    axis, cut = te.arrays(sp, D)
    G = te.growable(sp, p, n_cuts, D, 0.95, 2.0)
    P = te.prunable(sp)
    seen_grow, seen_prune = set(), set()
    u_grow, u_prune = 1 << 40, (2**64 - 1)
    for k in range(len(G)):
        w1 = (k * 2**32 + len(G) - 1) // len(G)
        eta = G[k]
        lo, hi = te.region(sp, eta, p, n_cuts)
        axes = [a for a in range(p) if hi[a] - lo[a] > 0]
        for ka, a in enumerate(axes):
            w1h = (ka * 2**32 + len(axes) - 1) // len(axes)
            avail = hi[a] - lo[a]
            for ks in range(avail):
                w2 = (ks * 2**32 + avail - 1) // avail
                out = oracle.propose(cfg, n_cuts, axis, cut, [u_grow, w1 | (w1h << 32), w2, 0])
                assert out[:4] == (1, eta, a, lo[a] + 1 + ks)
                assert out[4:] == (len(G), len(P))
                seen_grow.add(out[1:4])
    for k in range(len(P)):
        w1 = (k * 2**32 + len(P) - 1) // len(P)
        out = oracle.propose(cfg, n_cuts, axis, cut, [u_prune, w1, 0, 0])
        assert out[:2] == (2, P[k])
        seen_prune.add(out[1])
    assert len(seen_prune) == len(P)
    # a root-only tree always grows; a tree with no growable leaf prunes
    a0, c0 = te.arrays({}, D)
    assert oracle.propose(cfg, n_cuts, a0, c0, [2**64 - 1, 0, 0, 0])[0] == 1
    cfg0 = oracle.make_config(n=1, p=p, m=1, D=D, alpha=0.0, beta=2.0)
    assert oracle.propose(cfg0, n_cuts, a0, c0, [0, 0, 0, 0])[0] == 0
    assert oracle.propose(cfg0, n_cuts, axis, cut, [0, 0, 0, 0])[0] == 2


# --------------------------------------------------------------------------
# the Metropolis-Hastings kernel

def _tiny_problem(y_scale=1.0):
    p, n_cuts, D = 2, [2, 1], 3
    X = np.array([[0, 1, 2, 2, 0, 1], [1, 0, 1, 0, 0, 1]], np.uint8)
    y = y_scale * np.array([0.9, -0.4, 1.7, 1.2, -1.1, 0.3])
    return p, n_cuts, D, X, y


def _posterior(trees, X, y, sigma2, mu_mu, sigma_mu):
    lp = np.array([lp + te.log_marginal(sp, X, y, sigma2, mu_mu, sigma_mu)
                   for sp, lp in trees])
    w = np.exp(lp - lp.max())
    return w / w.sum()


@pytest.mark.parametrize("p_grow,alpha,beta,mu_mu", [(0.5, 0.95, 2.0, 0.0),
                                                     (0.3, 0.8, 0.5, 0.25),
                                                     (0.7, 0.6, 1.0, -0.4)])
def test_mh_kernel_leaves_posterior_invariant(p_grow, alpha, beta, mu_mu):
    """Exact transition matrix of GROW/PRUNE with the oracle's log r, for one
    tree at fixed sigma: pi_post K = pi_post, with pi_post computed by an
    independent route (prior x multivariate-normal marginal)."""
    p, n_cuts, D, X, y = _tiny_problem()
    sigma2, sigma_mu = 0.6, 0.7
    cfg = oracle.make_config(n=len(y), p=p, m=1, D=D, alpha=alpha, beta=beta, mu_mu=mu_mu,
                             sigma_mu=sigma_mu, p_grow=p_grow)
    trees = list(te.enumerate_trees(p, n_cuts, D, alpha, beta))
    index = {te.key(sp): k for k, (sp, _) in enumerate(trees)}
    post = _posterior(trees, X, y, sigma2, mu_mu, sigma_mu)
    K = np.zeros((len(trees), len(trees)))
    zeros = np.zeros(1 << D, np.float32)
    y32 = y.astype(np.float32)
    # the oracle's data pass sums fp32 residuals: use y rounded to fp32 on both
    post = _posterior(trees, X, y32.astype(np.float64), sigma2, mu_mu, sigma_mu)
    for k, (sp, _) in enumerate(trees):
        axis, cut = te.arrays(sp, D)
        idx_row = np.array([te.descend(sp, X, i) for i in range(len(y))], np.uint8)
        G, P = te.growable(sp, p, n_cuts, D, alpha, beta), te.prunable(sp)
        if not G and not P:
            K[k, k] = 1.0
            continue
        pg = 1.0 if not P else (0.0 if not G else p_grow)
        moves = []
        for eta in G:
            lo, hi = te.region(sp, eta, p, n_cuts)
            axes = [a for a in range(p) if hi[a] - lo[a] > 0]
            for a in axes:
                for s in range(lo[a] + 1, hi[a] + 1):
                    q = pg / len(G) / len(axes) / (hi[a] - lo[a])
                    new = dict(sp)
                    new[eta] = (a, s)
                    moves.append((q, 1, eta, a, s, new))
        for eta in P:
            new = dict(sp)
            del new[eta]
            moves.append(((1 - pg) / len(P), 2, eta, 0, 0, new))
        stay = 1.0
        for q, move, eta, a, s, new in moves:
            if q == 0:
                continue
            lr, _ = oracle.log_ratio(cfg, n_cuts, X, axis, cut, zeros, idx_row, y32, sigma2,
                                     move, eta, a, s)
            acc = min(1.0, math.exp(min(lr, 700.0)))
            K[k, index[te.key(new)]] += q * acc
            stay -= q * acc
        K[k, k] += stay
    np.testing.assert_allclose(K.sum(1), 1.0, atol=1e-14)
    np.testing.assert_allclose(post @ K, post, atol=1e-13, rtol=0)


def _chain_histogram(cfg, X, y, n_cuts, sigma2, seed, sweeps, burn=200):
    ch = oracle.Chain(cfg, X, n_cuts, y.astype(np.float32), sigma2)
    counts = {}
    ch.sweeps(seed, burn)
    H = 1 << (cfg.D - 1)
    for _ in range(sweeps):
        ch.run(seed, cfg.m + 1)
        sp = {}
        for h in range(1, H):
            if ch.cut[0, h] and (h == 1 or (h >> 1) in sp):
                sp[h] = (int(ch.axis[0, h]), int(ch.cut[0, h]))
        k = te.key(sp)
        counts[k] = counts.get(k, 0) + 1
    return counts


def test_chain_samples_tree_posterior():
    """The oracle's full sweep (proposal, data pass, accept, leaf draw,
    residual update), run as a chain with one tree and fixed sigma, visits
    trees with the posterior frequencies."""
    p, n_cuts, D, X, y = _tiny_problem()
    sigma2, sigma_mu, mu_mu = 0.6, 0.7, 0.1
    cfg = oracle.make_config(n=len(y), p=p, m=1, D=D, alpha=0.8, beta=0.5, mu_mu=mu_mu,
                             sigma_mu=sigma_mu, p_grow=0.5, fix_sigma2=True)
    trees = list(te.enumerate_trees(p, n_cuts, D, 0.8, 0.5))
    post = _posterior(trees, X, y.astype(np.float32).astype(np.float64), sigma2, mu_mu,
                      sigma_mu)
    N = 60000
    counts = _chain_histogram(cfg, X, y, n_cuts, sigma2, seed=99, sweeps=N)
    emp = np.array([counts.get(te.key(sp), 0) for sp, _ in trees]) / N
    assert sum(counts.values()) == N and len(counts) <= len(trees)
    tv = 0.5 * np.abs(emp - post).sum()
    assert tv < 0.03, (tv, emp, post)


def test_prior_only_chain_samples_tree_prior():
    """With y = 0 and a huge fixed sigma^2 the likelihood is flat: the chain
    samples the tree prior of sec. 2.1."""
    p, n_cuts, D, X, _ = _tiny_problem()
    y = np.zeros(X.shape[1])
    cfg = oracle.make_config(n=len(y), p=p, m=1, D=D, alpha=0.95, beta=1.0, mu_mu=0.0,
                             sigma_mu=0.5, fix_sigma2=True)
    trees = list(te.enumerate_trees(p, n_cuts, D, 0.95, 1.0))
    prior = np.array([math.exp(lp) for _, lp in trees])
    N = 60000
    counts = _chain_histogram(cfg, X, y, n_cuts, 1e10, seed=5, sweeps=N)
    emp = np.array([counts.get(te.key(sp), 0) for sp, _ in trees]) / N
    assert 0.5 * np.abs(emp - prior).sum() < 0.03


@pytest.mark.parametrize("m", [1, 3])
def test_no_split_model_is_normal_inverse_gamma(m):
    """alpha = 0: no tree can split and y_i = sum_j mu_j + eps_i.  The Gibbs
    chain over the m root leaves and sigma^2 must reproduce the posterior of
    (f = sum mu_j, sigma^2) under f ~ N(m mu_mu, m sigma_mu^2),
    sigma^2 ~ InvGamma(nu/2, nu lambda/2), computed by quadrature."""
    rng = np.random.default_rng(3)
    n = 12
    y = rng.normal(0.8, 1.1, n)
    mu_mu, sigma_mu, nu, lam = 0.1, 0.5, 3.0, 0.7
    X = np.zeros((1, n), np.uint8)
    cfg = oracle.make_config(n=n, p=1, m=m, D=3, alpha=0.0, beta=2.0, mu_mu=mu_mu,
                             sigma_mu=sigma_mu, nu=nu, lam=lam)
    ch = oracle.Chain(cfg, X, [3], y.astype(np.float32), 1.0)
    ch.sweeps(17, 100)
    fs, s2s = [], []
    for _ in range(40000):
        ch.run(17, m + 1)
        fs.append(float(ch.leaf[:, 1].astype(np.float64).sum()))
        s2s.append(ch.sigma2)
    fs, s2s = np.array(fs), np.array(s2s)
    y = y.astype(np.float32).astype(np.float64)
    prior_f = stats.norm(m * mu_mu, math.sqrt(m) * sigma_mu)
    prior_s = stats.invgamma(nu / 2.0, scale=nu * lam / 2.0)

    fg = np.linspace(-2.0, 3.5, 801)
    sg = np.linspace(0.05, 8.0, 1601)
    L = (prior_f.logpdf(fg)[:, None] + prior_s.logpdf(sg)[None, :]
         + stats.norm.logpdf(y[None, None, :], fg[:, None, None],
                             np.sqrt(sg)[None, :, None]).sum(-1))
    W = np.exp(L - L.max())
    W /= W.sum()
    Ef, Es = (W.sum(1) * fg).sum(), (W.sum(0) * sg).sum()
    sdf = math.sqrt((W.sum(1) * (fg - Ef) ** 2).sum())
    sds = math.sqrt((W.sum(0) * (sg - Es) ** 2).sum())
    # autocorrelated chain: allow an effective sample size of a few thousand
    assert abs(fs.mean() - Ef) < 6 * sdf / math.sqrt(4000), (fs.mean(), Ef)
    assert abs(s2s.mean() - Es) < 6 * sds / math.sqrt(4000), (s2s.mean(), Es)
    assert abs(fs.std() / sdf - 1) < 0.1 and abs(s2s.std() / sds - 1) < 0.15


# --------------------------------------------------------------------------
# whole sweeps on the small workload

@pytest.fixture(scope="module")
def small_chain():
    from paper_2410_23244_amd.inputs import make_inputs

    inp = make_inputs(1)
    h = inp.hyper
    cfg = oracle.make_config(n=inp.n, p=inp.p, m=inp.m, D=inp.D, alpha=h.alpha, beta=h.beta,
                             mu_mu=h.mu_mu, sigma_mu=h.sigma_mu, nu=h.nu, lam=h.lam,
                             p_grow=h.p_grow)
    ch = oracle.Chain(cfg, inp.X_b, inp.n_cuts, inp.y_c, h.sigma2_init)
    tr = ch.run(inp.seed, 60 * (inp.m + 1), trace=True)
    return inp, ch, tr


def test_cache_counts_and_residuals_stay_consistent(small_chain):
    inp, ch, tr = small_chain
    trees = tr[tr["kind"] == 0]
    # counts of the larger tree always cover every observation
    assert (trees["count"].sum(1) == inp.n).all()
    # the index cache equals Algorithm 1 on the current trees
    H = 1 << (inp.D - 1)
    for j in range(0, inp.m, 7):
        for i in range(0, inp.n, 37):
            assert ch.idx[j, i] == oracle.route(inp.D, ch.axis[j], ch.cut[j], inp.X_b, i)
    # residual cache vs y - sum of trees within the fp32 drift the paper quotes
    # (app. B: relative error ~1e-7 sqrt(n_tree) per iteration)
    f = ch.predict(inp.X_b, 0.0).astype(np.float64)
    err = np.abs(ch.resid.astype(np.float64) - (inp.y_c.astype(np.float64) - f)).max()
    k = 60
    assert err <= 10 * 1e-7 * math.sqrt(inp.m * k) * np.abs(inp.y_c).max(), err
    # nodes at depth D-1 never split and cut 0 marks leaves
    assert (ch.cut[:, : H][:, 0] == 0).all()


def test_sanity_bands(small_chain):
    inp, ch, tr = small_chain
    trees = tr[(tr["kind"] == 0) & (tr["sweep"] >= 20)]
    moved = trees[trees["move"] != 0]
    rate = moved["accept"].mean()
    assert 0.02 < rate < 0.6, rate        # sec. 2.2: typically 10-30 %
    leaves = trees["n_leaves"].mean()
    assert leaves < 10                     # sec. 2.2: at most ~10 leaves per tree
    sig = math.sqrt(tr[tr["kind"] == 1]["sigma2"][-20:].mean())
    assert 0.3 < sig < 0.8, sig            # noise sd of the workload is 0.5


def test_steps_compose_and_are_deterministic():
    from paper_2410_23244_amd.inputs import make_inputs

    inp = make_inputs(1, n=300, p=6, m=7)
    h = inp.hyper
    cfg = oracle.make_config(n=inp.n, p=inp.p, m=inp.m, D=inp.D, alpha=h.alpha, beta=h.beta,
                             mu_mu=h.mu_mu, sigma_mu=h.sigma_mu, nu=h.nu, lam=h.lam)
    a = oracle.Chain(cfg, inp.X_b, inp.n_cuts, inp.y_c, h.sigma2_init)
    b = oracle.Chain(cfg, inp.X_b, inp.n_cuts, inp.y_c, h.sigma2_init)
    a.sweeps(4, 3)
    a.sweeps(4, 2)
    b.run(4, 5 * (inp.m + 1) - 3)
    for _ in range(3):
        b.step(4)
    for name in ["axis", "cut", "leaf", "idx", "resid"]:
        np.testing.assert_array_equal(getattr(a, name), getattr(b, name))
    assert a.sigma2 == b.sigma2 and a.sweep == b.sweep == 5


def _numpy_philox_block(seed, ctr):
    prev = list(ctr)
    for k in range(4):
        prev[k] = (prev[k] - 1) % 2**64
        if ctr[k] != 0:
            break
    bg = np.random.Philox(key=np.array([seed, KEY_TAG], np.uint64),
                          counter=np.array(prev, np.uint64))
    return [int(w) for w in bg.random_raw(4)]


@pytest.mark.parametrize("chain", [0, 1, 37])
def test_chain_streams_offset_the_last_counter_word(chain):
    """Chain c draws block (s, j, q, c 2^32 + t): its accept uniform and leaf
    normals at sweep 0, tree 0 follow from numpy's Philox at that counter."""
    from paper_2410_23244_amd.inputs import make_inputs

    inp = make_inputs(1, n=300, p=6, m=3)
    h = inp.hyper
    seed = 9
    cfg = oracle.make_config(n=inp.n, p=inp.p, m=inp.m, D=inp.D, alpha=h.alpha, beta=h.beta,
                             mu_mu=h.mu_mu, sigma_mu=h.sigma_mu, nu=h.nu, lam=h.lam,
                             chain=chain)
    ch = oracle.Chain(cfg, inp.X_b, inp.n_cuts, inp.y_c, h.sigma2_init)
    tr = ch.step(seed)
    u01 = lambda w: ((w >> 12) + 0.5) * 2.0**-52
    w = _numpy_philox_block(seed, (0, 0, 0, chain << 32))
    assert tr["move"] == 1 and tr["eta"] == 1          # a root-only tree can only grow
    assert tr["ln_u"] == math.log(u01(w[3]))
    leaves = [2, 3] if tr["accept"] else [1]
    s2, sm2 = h.sigma2_init, h.sigma_mu ** 2
    for leaf in leaves:
        b = _numpy_philox_block(seed, (0, 0, 1, (chain << 32) + (leaf >> 1)))
        a, c = (b[2], b[3]) if leaf & 1 else (b[0], b[1])
        z = math.sqrt(-2.0 * math.log(u01(a))) * math.cos(2.0 * math.pi * u01(c))
        n_h = float(tr["count"][2] + tr["count"][3]) if leaf == 1 else float(tr["count"][leaf])
        S_h = float(tr["sum"][2] + tr["sum"][3]) if leaf == 1 else float(tr["sum"][leaf])
        prec = n_h / s2 + 1.0 / sm2
        want = (S_h / s2 + h.mu_mu / sm2) / prec + z / math.sqrt(prec)
        assert abs(tr["leaf_new"][leaf] - want) <= 1e-6 * (abs(want) + 1.0 / math.sqrt(prec))


def test_chains_are_independent_streams():
    from paper_2410_23244_amd.inputs import make_inputs

    inp = make_inputs(1, n=300, p=6, m=5)
    h = inp.hyper
    out = []
    for chain in [0, 1, 2]:
        cfg = oracle.make_config(n=inp.n, p=inp.p, m=inp.m, D=inp.D, alpha=h.alpha,
                                 beta=h.beta, mu_mu=h.mu_mu, sigma_mu=h.sigma_mu, nu=h.nu,
                                 lam=h.lam, chain=chain)
        ch = oracle.Chain(cfg, inp.X_b, inp.n_cuts, inp.y_c, h.sigma2_init)
        tr = ch.run(4, 3 * (inp.m + 1), trace=True)
        out.append((tr["ln_u"].copy(), ch.sigma2))
    for a in range(3):
        for b in range(a + 1, 3):
            assert not np.array_equal(out[a][0], out[b][0])
            assert out[a][1] != out[b][1]


# --------------------------------------------------------------------------
# probit model (binary y by latent normals)

def test_normal_cdf_and_inverse():
    # the tail is conditioned like x^2 eps in the argument of erfc
    x = np.concatenate([np.linspace(-37, 8, 400), [0.0]])
    np.testing.assert_allclose([oracle.norm_cdf(v) for v in x], stats.norm.cdf(x),
                               rtol=2e-16 * (1 + 37.0**2), atol=0)
    p = np.concatenate([np.logspace(-300, -1, 150), np.linspace(0.01, 0.99, 99),
                        [1 - 1e-12, 1 - 2**-53]])
    got = np.array([oracle.norm_ppf(v) for v in p])
    np.testing.assert_allclose(got, stats.norm.ppf(p), rtol=2e-15, atol=2e-15)


@pytest.mark.parametrize("f", [-3.0, -0.4, 0.0, 1.7, 6.0])
def test_latent_draw_is_the_truncated_normal_quantile(f):
    """z | f, y is N(f, 1) truncated to z <= 0 (y = 0) or z > 0 (y = 1); the
    draw at uniform u is that law's quantile (at u for y = 0, at 1 - u for
    y = 1, the reflected inversion)."""
    u = np.linspace(0.001, 0.999, 57)
    lo = stats.truncnorm(-np.inf, -f, loc=f)
    hi = stats.truncnorm(-f, np.inf, loc=f)
    z0 = np.array([oracle.latent_draw(f, 0, v) for v in u])
    z1 = np.array([oracle.latent_draw(f, 1, v) for v in u])
    assert (z0 <= 0).all() and (z1 > 0).all()
    np.testing.assert_allclose(z0, lo.ppf(u), rtol=1e-9, atol=1e-9)
    np.testing.assert_allclose(z1, hi.ppf(1 - u), rtol=1e-9, atol=1e-9)


@pytest.mark.parametrize("m", [1, 3])
def test_probit_no_split_model_matches_quadrature(m):
    """alpha = 0: y_i ~ Bernoulli(Phi(offset + sum_j mu_j)).  The latent Gibbs
    chain over the m root leaves must reproduce the posterior of
    f = sum mu_j under f ~ N(m mu_mu, m sigma_mu^2), by quadrature."""
    rng = np.random.default_rng(5)
    n = 30
    yb = (rng.random(n) < 0.7).astype(np.float32)
    mu_mu, sigma_mu, off = 0.05, 0.6, 0.2
    X = np.zeros((1, n), np.uint8)
    cfg = oracle.make_config(n=n, p=1, m=m, D=3, alpha=0.0, beta=2.0, mu_mu=mu_mu,
                             sigma_mu=sigma_mu, probit=True, probit_offset=off)
    ch = oracle.Chain(cfg, X, [3], yb, 1.0)
    assert ch.sigma2 == 1.0
    ch.sweeps(23, 200)
    fs = []
    for _ in range(40000):
        ch.run(23, m + 1)
        fs.append(float(ch.leaf[:, 1].astype(np.float64).sum()))
        assert ((ch.latent > 0) == (yb > 0)).all()
    fs = np.array(fs)
    assert ch.sigma2 == 1.0
    fg = np.linspace(-4.0, 4.0, 4001)
    k = int(yb.sum())
    L = (stats.norm(m * mu_mu, math.sqrt(m) * sigma_mu).logpdf(fg)
         + k * stats.norm.logcdf(off + fg) + (n - k) * stats.norm.logcdf(-(off + fg)))
    W = np.exp(L - L.max())
    W /= W.sum()
    Ef = (W * fg).sum()
    sdf = math.sqrt((W * (fg - Ef) ** 2).sum())
    assert abs(fs.mean() - Ef) < 6 * sdf / math.sqrt(4000), (fs.mean(), Ef)
    assert abs(fs.std() / sdf - 1) < 0.1, (fs.std(), sdf)


def test_probit_chain_recovers_class_probabilities():
    """Binary data from P(y = 1 | x) = Phi(g(x)); the posterior mean of
    Phi(f) tracks the true probabilities."""
    from paper_2410_23244_amd.inputs import bin_column, cutpoints

    rng = np.random.default_rng(8)
    n, p, m = 3000, 4, 50
    X = rng.random((p, n)).astype(np.float32)
    g = 1.5 * np.sin(2 * np.pi * X[0]) + 2.0 * (X[1] - 0.5)
    yb = (rng.random(n) < stats.norm.cdf(g)).astype(np.float32)
    Xb = np.stack([bin_column(X[a], cutpoints(X[a], 63, "quantile")) for a in range(p)])
    off = float(stats.norm.ppf(yb.mean()))
    cfg = oracle.make_config(n=n, p=p, m=m, D=6, mu_mu=0.0, sigma_mu=3.0 / (2 * math.sqrt(m)),
                             probit=True, probit_offset=off)
    ch = oracle.Chain(cfg, Xb, np.full(p, 63, np.int32), yb, 1.0)
    ch.sweeps(4, 200)
    acc = np.zeros(n)
    for _ in range(200):
        ch.sweeps(4, 1)
        acc += stats.norm.cdf(ch.predict(Xb, off).astype(np.float64))
    prob = acc / 200
    err = np.abs(prob - stats.norm.cdf(g))
    assert err.mean() < 0.06, err.mean()
    # beats the constant predictor by far
    assert err.mean() < 0.3 * np.abs(yb.mean() - stats.norm.cdf(g)).mean()
