"""Lockstep comparison of the HIP sweep with the CPU oracle.

The device chain runs to some state, the oracle loads that state, then both
execute the same steps (tree steps and sigma^2 steps, same seed) and every
step's record is compared:

* move, node, axis, cut, #G(T), #P(T), every per-leaf count: bit-exact;
* accept: bit-exact, except a tie |ln u - log r| <= 1e-4 (1 + sum |terms|),
  where the oracle adopts the device decision to stay in lockstep;
* partial-residual sums S_h: |dS| <= 1e-5 x the leaf's l1 mass
  sum_i |r_i| + n_h |old value| (sums cancel, so relative error is measured
  against the mass that was summed);
* new leaf values: |dmu| <= 1e-5 (|mu| + 1/sqrt(prec));
* SSR and sigma^2: relative 1e-5 (the device sums fp32 workgroup partials);
and at the end the index caches and tree structures must be identical and
the residuals close.  After each tree step the oracle carries on from the
device's new leaf values (and, on a tie, its decision), so that every step
compares the two implementations on identical trees, residuals and random
streams rather than on two chains that drift apart by fp32 rounding.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

import oracle


@dataclass
class Report:
    steps: int = 0
    tree_steps: int = 0
    accepts: int = 0
    ties: int = 0
    moves: int = 0
    max_sum_err: float = 0.0      # max |dS| / l1 mass (an upper bound: |dS| / |S| where
                                  # that already meets the tolerance)
    max_leaf_err: float = 0.0     # max |dmu| / (|mu| + 1/sqrt(prec))
    max_logr_err: float = 0.0
    max_resid_err: float = 0.0
    notes: list = field(default_factory=list)


def chain_from_state(inp, st, chain=0) -> oracle.Chain:
    return oracle.chain_from_state(inp, st, chain=chain)


def _leaf_l1(inp, idx_row, resid, leaf_row, move, eta, a, s):
    """l1 mass of the partial residuals of every larger-tree leaf (256 slots)."""
    c = idx_row.astype(np.int64)
    cp = c.copy()
    if move == 1:
        sel = c == eta
        cp[sel] = 2 * eta + (inp.X_b[a][sel] >= s)
    l1 = np.bincount(cp, weights=np.abs(resid.astype(np.float64)), minlength=256)
    cnt = np.bincount(cp, minlength=256).astype(np.float64)
    old = np.zeros(256)
    old[: leaf_row.size] = np.abs(leaf_row.astype(np.float64))
    if move == 1:
        old[2 * eta] = old[eta]
        old[2 * eta + 1] = old[eta]
    return l1 + cnt * old


def compare_steps(inp, ch: oracle.Chain, trg: np.ndarray, seed: int, rep: Report,
                  sum_tol=1e-5, leaf_tol=1e-5, tie_tol=1e-4, var_tol=1e-5, adopt_leaves=True):
    H = 1 << (inp.D - 1)
    sig_mu2 = inp.hyper.sigma_mu ** 2
    for k, g in enumerate(trg):
        rep.steps += 1
        j = ch.next
        if j < inp.m:
            saved = (ch.idx[j].copy(), ch.resid.copy(), ch.axis[j].copy(), ch.cut[j].copy(),
                     ch.leaf[j].copy(), ch.sigma2, ch.sweep, ch.next)
            # the oracle continues from the device's leaf draws (compared below), so every
            # step starts from identical trees, residuals and random streams
            adopt = g["leaf_new"] if adopt_leaves else None
            o = ch.step(seed, adopt=adopt)
            assert g["kind"] == 0 and o["kind"] == 0, (k, g["kind"], o["kind"])
            assert (g["tree"], g["sweep"]) == (o["tree"], o["sweep"]), (k, g["tree"], o["tree"])
            for f in ["move", "eta", "axis", "cut", "n_grow_cand", "n_prune_cand", "n_leaves"]:
                assert g[f] == o[f], (k, j, f, g[f], o[f])
            np.testing.assert_array_equal(g["count"], o["count"], err_msg=f"counts step {k}")
            rep.tree_steps += 1
            if o["move"] != 0:
                rep.moves += 1
                band = tie_tol * (1.0 + o["log_r_scale"])
                rep.max_logr_err = max(rep.max_logr_err, abs(g["log_r"] - o["log_r"]) / band)
                assert abs(g["ln_u"] - o["ln_u"]) <= 1e-12 * (1 + abs(o["ln_u"])), k
                if g["accept"] != o["accept"]:
                    if abs(o["ln_u"] - o["log_r"]) > band:
                        raise AssertionError(f"step {k} tree {j}: accept gpu={g['accept']} "
                                             f"oracle={o['accept']} ln_u={o['ln_u']} "
                                             f"log_r={o['log_r']} gpu log_r={g['log_r']}")
                    rep.ties += 1
                    rep.notes.append(f"tie at step {k} (tree {j})")
                    (ch.idx[j], ch.resid[...], ch.axis[j], ch.cut[j], ch.leaf[j]) = (
                        saved[0], saved[1], saved[2], saved[3], saved[4])
                    ch.sigma2, ch.sweep, ch.next = saved[5], saved[6], saved[7]
                    o = ch.step(seed, force=int(g["accept"]), adopt=adopt)
                rep.accepts += int(o["accept"])
            # partial-residual sums against the l1 mass of each leaf.  |S_h| is
            # at most that mass, so a sum within sum_tol |S_h| passes without it;
            # the mass itself (a pass over the data) is formed only for leaves
            # whose sums cancel
            used = o["count"] > 0
            err = np.abs(g["sum"] - o["sum"])
            rel = np.where(used, err / np.maximum(np.abs(o["sum"]), 1e-300), err)
            if rel.max() > sum_tol:
                l1 = _leaf_l1(inp, saved[0], saved[1], saved[4], int(o["move"]),
                              int(o["eta"]), int(o["axis"]), int(o["cut"]))
                rel = np.where(used, err / np.maximum(l1, 1e-30), err)
            rep.max_sum_err = max(rep.max_sum_err, float(rel.max()))
            assert rel.max() <= sum_tol, (k, j, float(rel.max()))
            # new leaf values
            cnt = o["count"].astype(np.float64)
            if (o["move"] == 1 and not o["accept"]) or (o["move"] == 2 and o["accept"]):
                e = int(o["eta"])
                cnt[e] = cnt[2 * e] + cnt[2 * e + 1]
            prec = cnt / o["sigma2"] + 1.0 / sig_mu2
            scale = np.abs(o["leaf_new"].astype(np.float64)) + 1.0 / np.sqrt(prec)
            lerr = np.abs(g["leaf_new"].astype(np.float64) - o["leaf_new"]) / scale
            rep.max_leaf_err = max(rep.max_leaf_err, float(lerr.max()))
            assert lerr.max() <= leaf_tol, (k, j, float(lerr.max()))
        else:
            o = ch.step(seed)
            assert g["kind"] == 1 and o["kind"] == 1, (k, g["kind"], o["kind"])
            assert g["sweep"] == o["sweep"]
            assert abs(g["ssr"] - o["ssr"]) <= var_tol * o["ssr"], (k, g["ssr"], o["ssr"])
            assert abs(g["sigma2"] - o["sigma2"]) <= var_tol * o["sigma2"], (k, g["sigma2"],
                                                                           o["sigma2"])
            # keep the chains on the same sigma^2 so the next sweep is comparable
            ch.sigma2 = float(g["sigma2"])
    return rep


def compare_states(inp, gst: dict, ch: oracle.Chain, rep: Report):
    np.testing.assert_array_equal(gst["idx"], ch.idx, err_msg="index cache")
    np.testing.assert_array_equal(gst["cut"], ch.cut, err_msg="cut")
    H = 1 << (inp.D - 1)
    for j in range(inp.m):
        for h in range(1, H):
            if gst["cut"][j, h]:
                assert gst["axis"][j, h] == ch.axis[j, h], (j, h)
    # the oracle adopted the device's leaf draws, so the fp32 residual updates
    # r + (old - new) were the same operations on the same values on both sides
    rep.max_resid_err = float(np.abs(gst["resid"].astype(np.float64) - ch.resid).max())
    if getattr(inp, "probit", False):
        # the latent draws invert the normal cdf with each side's own
        # implementation (fp64, a few ulps apart) before rounding to f32
        tol = 1e-6 * (1.0 + np.abs(ch.latent.astype(np.float64)))
        assert (np.abs(gst["latent"].astype(np.float64) - ch.latent) <= tol).all(), "latents"
        assert ((gst["latent"] > 0) == (ch.ybin > 0)).all()
        tol = 1e-6 * (1.0 + np.abs(ch.resid.astype(np.float64)))
        assert (np.abs(gst["resid"].astype(np.float64) - ch.resid) <= tol).all(), "residuals"
    else:
        np.testing.assert_array_equal(gst["resid"], ch.resid, err_msg="residual cache")
    np.testing.assert_array_equal(gst["leaf"], ch.leaf, err_msg="leaf values")
    assert gst["sweep"] == ch.sweep and gst["next"] == ch.next
    assert abs(gst["sigma2"] - ch.sigma2) <= 1e-5 * ch.sigma2


def lockstep(inp, gpu, seed: int, warm_sweeps: int, n_steps: int) -> Report:
    """Warm the device chain, then run n_steps in lockstep with the oracle."""
    return lockstep_chains(inp, gpu, seed, warm_sweeps, n_steps)[0]


def lockstep_chains(inp, gpu, seed: int, warm_sweeps: int, n_steps: int) -> list:
    """lockstep for every chain of the handle: chain c against an oracle chain
    drawing from stream c."""
    C = gpu.nchain
    if warm_sweeps:
        gpu.step(warm_sweeps, seed)
    chs = [chain_from_state(inp, gpu.get_state(c), chain=c) for c in range(C)]
    assert gpu.status() == 0
    trg = gpu.debug_steps(n_steps, seed)
    assert gpu.status() == 0
    trg = trg.reshape(C, n_steps)
    reps = []
    for c in range(C):
        rep = compare_steps(inp, chs[c], trg[c], seed, Report())
        compare_states(inp, gpu.get_state(c), chs[c], rep)
        reps.append(rep)
    return reps


def leaf_slots(cut_row: np.ndarray) -> np.ndarray:
    """Leaves of one heap tree (cut row u8 [H]) as a mask over its 2H slots:
    present slots (the root, and children of a split node above the last
    level) that do not split."""
    H = cut_row.size
    present = np.zeros(2 * H, bool)
    present[1] = True
    for h in range(2, 2 * H):
        present[h] = present[h >> 1] and cut_row[h >> 1] != 0
    return present & np.concatenate([cut_row == 0, np.ones(H, bool)])


def check_invariants(inp, st: dict, sweeps: int, n_sample: int = 256, seed: int = 0) -> dict:
    """What must hold of any state the device reaches, traced or not (sec. 3.3
    "Traverse indices cache" and "Residuals cache", app. B):
    * the index cache holds each observation's leaf: on a sample of points,
      every tree's entry equals the oracle's descent of that tree;
    * the per-leaf counts the sampler keeps sum to n over the leaves of every
      tree and equal the histogram of the tree's index row (slots that are
      not leaves keep stale counts, which nothing reads);
    * the residual cache equals y_c minus the sum of trees up to the drift of
      fp32 updates: ||r - (y_c - sum_j mu_j[idx_j])||_inf / max|y_c| <=
      10 * 1e-7 * sqrt(m * sweeps).
    Returns the measured quantities."""
    n, m, H = inp.n, inp.m, 1 << (inp.D - 1)
    idx = st["idx"].reshape(m, n)
    rng = np.random.default_rng(seed)
    sample = rng.choice(n, size=min(n_sample, n), replace=False)
    for j in range(m):
        for i in sample:
            want = oracle.route(inp.D, st["axis"][j], st["cut"][j], inp.X_b, int(i))
            assert idx[j, i] == want, (j, int(i), int(idx[j, i]), want)
    cnt = st["count"].reshape(m, 2 * H)
    for j in range(m):
        # leaves of tree j: present slots (the root, and children of a split
        # node above the last level) that do not split
        is_leaf = leaf_slots(st["cut"][j])
        hist = np.bincount(idx[j], minlength=2 * H)[: 2 * H]
        assert hist[~is_leaf].sum() == 0, f"index entries off the leaves of tree {j}"
        assert cnt[j][is_leaf].sum() == n, f"counts of tree {j} do not sum to n"
        np.testing.assert_array_equal(cnt[j][is_leaf], hist[is_leaf], err_msg=f"counts tree {j}")
    f = np.zeros(n)
    leaf = st["leaf"].astype(np.float64)
    for j in range(m):
        f += leaf[j][idx[j]]
    drift = float(np.abs(st["resid"].astype(np.float64) - (inp.y_c[:n].astype(np.float64) - f)).max())
    scale = float(np.abs(inp.y_c[:n]).max())
    bound = 10 * 1e-7 * math.sqrt(m * max(sweeps, 1))
    assert drift <= bound * scale, (drift, bound * scale)
    return {"route_checked": int(len(sample) * m), "resid_drift": drift / scale, "bound": bound}
