"""Brute-force tree helpers for the oracle pins, written independently of the
oracle: recursive enumeration of every heap tree allowed by a tiny grid, the
generative tree prior of sec. 2.1 evaluated node by node while enumerating,
recursive descent, and the multivariate-normal marginal likelihood of the
data under a tree with its leaves integrated out."""
from __future__ import annotations

import itertools
import math

import numpy as np
from scipy.stats import multivariate_normal


def enumerate_trees(p, n_cuts, D, alpha, beta):
    """All trees of maximum depth D on the grid n_cuts.  Yields
    (splits, log_prior) where splits maps heap index -> (axis, cut) for the
    internal nodes.  The prior is the generative one: a node at depth d with
    at least one available split is internal with probability
    alpha (1+d)^-beta, then draws its axis uniformly among the axes with an
    available split and its cut uniformly among those."""
    H = 1 << (D - 1)

    def rec(h, lo, hi):
        d = int(math.floor(math.log2(h)))
        axes = [a for a in range(p) if hi[a] - lo[a] > 0]
        can = (h < H) and len(axes) > 0
        ps = alpha * (1.0 + d) ** (-beta) if can else 0.0
        out = [({}, math.log1p(-ps) if ps < 1 else -math.inf)]
        if not can or ps == 0.0:
            return out
        for a in axes:
            for s in range(lo[a] + 1, hi[a] + 1):
                lp_node = math.log(ps) - math.log(len(axes)) - math.log(hi[a] - lo[a])
                hl = list(hi)
                hl[a] = s - 1
                lr = list(lo)
                lr[a] = s
                for (sl, lpl), (sr, lpr) in itertools.product(rec(2 * h, lo, hl),
                                                              rec(2 * h + 1, lr, hi)):
                    sp = {h: (a, s)}
                    sp.update(sl)
                    sp.update(sr)
                    out.append((sp, lp_node + lpl + lpr))
        return out

    yield from rec(1, [0] * p, list(n_cuts))


def arrays(splits, D):
    H = 1 << (D - 1)
    axis = np.zeros(H, np.uint16)
    cut = np.zeros(H, np.uint8)
    for h, (a, s) in splits.items():
        axis[h] = a
        cut[h] = s
    return axis, cut


def key(splits):
    return tuple(sorted(splits.items()))


def descend(splits, X, i):
    h = 1
    while h in splits:
        a, s = splits[h]
        h = 2 * h + (1 if X[a, i] >= s else 0)
    return h


def leaves(splits):
    out, stack = [], [1]
    while stack:
        h = stack.pop()
        if h in splits:
            stack += [2 * h, 2 * h + 1]
        else:
            out.append(h)
    return sorted(out)


def region(splits, h, p, n_cuts):
    lo, hi = [0] * p, list(n_cuts)
    path = []
    while h > 1:
        path.append(h)
        h >>= 1
    for c in reversed(path):
        a, s = splits[c >> 1]
        if c & 1:
            lo[a] = s
        else:
            hi[a] = s - 1
    return lo, hi


def growable(splits, p, n_cuts, D, alpha, beta):
    """Leaves with a positive split probability, increasing heap order."""
    out = []
    for h in leaves(splits):
        d = int(math.floor(math.log2(h)))
        lo, hi = region(splits, h, p, n_cuts)
        if d < D - 1 and any(hi[a] - lo[a] > 0 for a in range(p)) and alpha > 0:
            out.append(h)
    return out


def prunable(splits):
    return sorted(h for h in splits if 2 * h not in splits and 2 * h + 1 not in splits)


def log_marginal(splits, X, y, sigma2, mu_mu, sigma_mu):
    """log N(y; mu_mu 1, sigma^2 I + sigma_mu^2 Z Z^T), Z the leaf indicators."""
    n = len(y)
    lv = [descend(splits, X, i) for i in range(n)]
    Z = np.array([[1.0 if lv[i] == h else 0.0 for h in leaves(splits)] for i in range(n)])
    cov = sigma2 * np.eye(n) + sigma_mu**2 * Z @ Z.T
    return float(multivariate_normal(mean=np.full(n, mu_mu), cov=cov).logpdf(y))
