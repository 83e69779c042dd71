"""Parity of the HIP sweep (through the C ABI) with the CPU oracle, lockstep.

Small cases cover every workload shape (u8 and u16 index caches, depth 6 and
8, one and many workgroups, ragged tails); the full-size cases run the
headline shapes in the launch configuration the benchmark times."""
from __future__ import annotations

import functools

import numpy as np
import pytest

from paper_2410_23244_amd.inputs import make_inputs
from tests import parity

pytestmark = pytest.mark.gpu


COOP, ORDINARY = 0, 1  # BART_LAUNCH_COOPERATIVE, BART_LAUNCH_ORDINARY
AUTO, REGS, STREAM = 0, 1, 2  # BART_RESID_AUTO, BART_RESID_REGISTERS, BART_RESID_STREAMED


@functools.lru_cache(maxsize=None)
def _full(cfg):
    """A full-size workload, generated once per test session (the large ones
    take tens of seconds); the tests that use it do not modify it."""
    return make_inputs(cfg)


def _gpu(inp, grid=0, launch=COOP, residency=AUTO, nchain=1):
    from paper_2410_23244_amd.bart import from_inputs

    return from_inputs(inp, grid=grid, launch=launch, residency=residency, nchain=nchain)


CASES = {
    # name: (config, overrides, warm sweeps, lockstep steps, grid, launch[, residency])
    "w1_full": (1, dict(), 3, 2 * 51, 0, COOP),
    "w1_ragged_tiny": (1, dict(n=37, p=3, m=5), 2, 3 * 6, 0, COOP),
    "w2_ragged": (2, dict(n=20011, m=60), 2, 61 + 30, 0, COOP),
    "w2_many_wg": (2, dict(n=40003, p=30, m=40), 2, 41 * 2, 10, ORDINARY),
    "w2_idle_wg": (2, dict(n=20011, p=30, m=30), 2, 31 * 2, 8, COOP),
    "w4_u16": (4, dict(n=30001, p=20, m=50), 2, 51 + 10, 0, COOP),
    "w5_depth8": (5, dict(n=25003, p=1000, m=120), 2, 121 + 5, 0, COOP),
    # residuals streamed from HBM: ragged chunks per thread, u16 cache, depth 8
    "w2_stream": (2, dict(n=40003, p=30, m=40), 2, 41 * 2, 4, ORDINARY, STREAM),
    "w1_stream_tiny": (1, dict(n=37, p=3, m=5), 2, 3 * 6, 0, COOP, STREAM),
    "w1_stream_one_wg": (1, dict(n=997, p=8, m=12), 2, 13 * 2, 1, ORDINARY, STREAM),
    "w4_stream_u16": (4, dict(n=70001, p=20, m=50), 2, 51 + 10, 0, COOP, STREAM),
    "w5_stream_depth8": (5, dict(n=25003, p=1000, m=120), 2, 121 + 5, 3, COOP, STREAM),
    # degenerate shapes: one observation, one chunk and a point, the shallowest
    # trees (a root and its two children), a single tree, a single predictor
    "w1_one_point": (1, dict(n=1, p=2, m=3), 2, 4 * 3, 0, COOP),
    "w1_five_points_stream": (1, dict(n=5, p=3, m=4), 2, 5 * 3, 0, COOP, STREAM),
    "w1_depth2": (1, dict(n=301, p=3, m=4, D=2), 2, 5 * 4, 0, COOP),
    "w2_one_tree": (2, dict(n=5003, p=10, m=1), 3, 2 * 20, 0, COOP),
    "w2_one_tree_stream": (2, dict(n=5003, p=10, m=1), 3, 2 * 20, 0, COOP, STREAM),
    "w2_one_tree_no_cache": (2, dict(n=5003, p=10, m=1, idx_bytes=0), 3, 2 * 20, 0, COOP, STREAM),
    "w2_two_trees_no_cache": (2, dict(n=5003, p=10, m=2, idx_bytes=0), 3, 3 * 12, 0, ORDINARY,
                              STREAM),
    "w2_one_axis": (2, dict(n=2000, p=1, m=3), 2, 4 * 5, 0, ORDINARY),
}


@pytest.mark.parametrize("name", list(CASES))
def test_lockstep_small(name):
    cfg, over, warm, steps, grid, launch, *rest = CASES[name]
    residency = rest[0] if rest else AUTO
    inp = make_inputs(cfg, **over)
    print(f"case {name}: n={inp.n} p={inp.p} m={inp.m} D={inp.D} idx={inp.idx_bytes}", flush=True)
    g = _gpu(inp, grid, launch, residency)
    info = g.launch_info()
    print(f"  grid={info.grid} chunks/thread={info.chunks_per_thread} "
          f"residency={info.residency}", flush=True)
    if residency == STREAM:
        assert info.residency == STREAM and info.rank_stash == 1
    rep = parity.lockstep(inp, g, seed=inp.seed + 100, warm_sweeps=warm, n_steps=steps)
    print(f"  {rep}", flush=True)
    assert rep.tree_steps > 0 and rep.moves > 0


def test_predict_matches_oracle():
    inp = make_inputs(1, n=3001, p=10, m=30)
    g = _gpu(inp)
    g.step(5, 7)
    st = g.get_state()
    ch = parity.chain_from_state(inp, st)
    Xt = make_inputs(1, n=1999, p=10, m=30).X_b
    want = ch.predict(Xt, inp.offset)
    got = g.predict(Xt, inp.offset).cpu().numpy()
    np.testing.assert_array_equal(got, want)
    # on the training set, y_c - f equals the residual cache up to fp32 drift
    f = g.predict(inp.X_b, 0.0).cpu().numpy().astype(np.float64)
    err = np.abs(st["resid"] - (inp.y_c.astype(np.float64) - f)).max()
    assert err < 1e-4 * np.abs(inp.y_c).max()


def test_steps_compose_and_are_deterministic():
    inp = make_inputs(2, n=5003, p=12, m=9)
    a, b = _gpu(inp), _gpu(inp)
    a.step(3, 11)
    a.step(2, 11)
    b.step(5, 11)
    sa, sb = a.get_state(), b.get_state()
    for k in ["axis", "cut", "leaf", "idx", "resid"]:
        np.testing.assert_array_equal(sa[k], sb[k], err_msg=k)
    assert sa["sigma2"] == sb["sigma2"] and sa["sweep"] == sb["sweep"] == 5


def test_set_state_roundtrip_continues_identically():
    # n = 2001: the last chunk of 4 points holds one point and three padding
    inp = make_inputs(1, n=2001, p=8, m=12)
    a = _gpu(inp)
    a.step(4, 3)
    st = a.get_state()
    b = _gpu(inp)
    b.set_state(st)
    a.step(2, 3)
    b.step(2, 3)
    sa, sb = a.get_state(), b.get_state()
    for k in ["axis", "cut", "leaf", "idx", "resid"]:
        np.testing.assert_array_equal(sa[k], sb[k], err_msg=k)
    assert a.status() == 0 and b.status() == 0


def test_set_state_flags_an_inconsistent_index_cache():
    """Index entry 0 marks a padding point; a real point whose entry is 0
    (or any slot outside 1..2H-1) makes the leaf recount that set_state runs
    report an inconsistent cache (BART_DEVERR_CACHE = 2)."""
    inp = make_inputs(1, n=2001, p=8, m=12)
    a = _gpu(inp)
    a.step(3, 3)
    st = a.get_state()
    assert a.status() == 0
    for bad_value in (0, 1 << (inp.D - 1 + 1)):
        bad = dict(st)
        bad["idx"] = st["idx"].copy()
        bad["idx"][3, 17] = bad_value
        b = _gpu(inp)
        b.set_state(bad)
        assert b.status() == 2, bad_value
    c = _gpu(inp)
    c.set_state(st)
    assert c.status() == 0


@pytest.mark.parametrize("residency", [REGS, STREAM])
def test_an_absent_workgroup_ends_the_launch_with_a_timeout(residency):
    """Every cross-workgroup wait is bounded: with one workgroup of the grid
    left out and a small spin limit, the launch returns and reports
    BART_DEVERR_TIMEOUT (1) instead of waiting for it; the workgroups that
    ran exit normally, and a new chain on the same inputs then runs clean."""
    inp = make_inputs(2, n=20011, p=10, m=12)
    g = _gpu(inp, launch=ORDINARY, residency=residency)
    info = g.launch_info()
    print(f"grid={info.grid} residency={info.residency}", flush=True)
    assert info.grid >= 2
    g.debug_stall(2 * (inp.m + 1), 5, 1, 2000)
    assert g.status() & 1
    g.close()
    h = _gpu(inp, launch=ORDINARY, residency=residency)
    h.step(2, 5)
    assert h.status() == 0


def test_launch_modes_agree():
    inp = make_inputs(2, n=30011, p=16, m=20)
    a, b = _gpu(inp, launch=COOP), _gpu(inp, launch=ORDINARY)
    assert a.launch_info().launch == COOP and b.launch_info().launch == ORDINARY
    a.step(6, 5)
    b.step(6, 5)
    sa, sb = a.get_state(), b.get_state()
    for k in ["axis", "cut", "leaf", "idx", "resid"]:
        np.testing.assert_array_equal(sa[k], sb[k], err_msg=k)
    assert sa["sigma2"] == sb["sigma2"]


@pytest.mark.parametrize("cfg", [2, 3, 5])
def test_lockstep_full_size(cfg):
    """Full size, in the launch mode the benchmark times, after the benchmark's
    warm-up length (trees near their stationary size): the untraced warm-up
    leaves a state that meets the cache invariants, then a whole sweep runs
    in lockstep with the oracle."""
    inp = _full(cfg)
    print(f"full workload {cfg}: n={inp.n} p={inp.p} m={inp.m}", flush=True)
    g = _gpu(inp, launch=ORDINARY)
    g.step(100, inp.seed)
    assert g.status() == 0
    inv = parity.check_invariants(inp, g.get_state(), sweeps=100)
    print(f"  invariants after 100 untraced sweeps: {inv}", flush=True)
    rep = parity.lockstep(inp, g, seed=inp.seed, warm_sweeps=0, n_steps=inp.m + 1)
    print(f"  {rep}", flush=True)


# sweeps in lockstep from the initial state (root-only trees, where GROW
# dominates): every sweep of the tiny workload, ten of workload 2, two of the
# large ones
FROM_INIT = {1: 100, 2: 10, 3: 2, 4: 2, 5: 2}


@pytest.mark.parametrize("cfg", sorted(FROM_INIT))
def test_lockstep_from_init(cfg):
    inp = _full(cfg)
    k = FROM_INIT[cfg]
    print(f"workload {cfg} from init: n={inp.n} p={inp.p} m={inp.m}, {k} sweeps", flush=True)
    g = _gpu(inp, launch=ORDINARY)
    rep = parity.lockstep(inp, g, seed=inp.seed, warm_sweeps=0, n_steps=k * (inp.m + 1))
    print(f"  {rep}", flush=True)
    assert rep.tree_steps == k * inp.m and rep.moves > 0


@pytest.mark.parametrize("cfg", [3, 4, 5])
def test_timed_path_equals_traced_path(cfg):
    """bart_step (no trace: the call bench.py times) and bart_debug_steps (the
    call the lockstep tests compare with the oracle) from one state give the
    same chain bit for bit, at full size in the benchmark's launch mode."""
    inp = _full(cfg)
    g = _gpu(inp, launch=ORDINARY)
    g.step(3, inp.seed)
    s0 = g.get_state()
    g.step(2, inp.seed)
    a = g.get_state()
    g.set_state(s0)
    g.debug_steps(2 * (inp.m + 1), inp.seed)
    b = g.get_state()
    assert g.status() == 0
    for key in ["axis", "cut", "leaf", "idx", "resid"]:
        np.testing.assert_array_equal(a[key], b[key], err_msg=key)
    # the counts of the leaves (set_state recounted b's from the index cache,
    # so slots that are no longer leaves differ: nothing reads them)
    for j in range(inp.m):
        lv = parity.leaf_slots(a["cut"][j])
        np.testing.assert_array_equal(a["count"][j][lv], b["count"][j][lv], err_msg=f"count {j}")
    assert a["sigma2"] == b["sigma2"] and a["sweep"] == b["sweep"] == s0["sweep"] + 2


def _full_trees(inp, depth, rng):
    """A state whose trees are all complete to `depth` (2**depth leaves), with
    random axes, cuts and leaf values, the index cache routed by brute force
    and residuals y_c - sum of trees."""
    m, H, n, p = inp.m, 1 << (inp.D - 1), inp.n, inp.p
    axis = np.zeros((m, H), np.uint16)
    cut = np.zeros((m, H), np.uint8)
    leaf = np.zeros((m, 2 * H), np.float32)
    idx = np.zeros((m, n), np.uint8 if inp.idx_bytes == 1 else np.uint16)
    f = np.zeros(n)
    for j in range(m):
        for h in range(1, 1 << depth):
            # region of h: the ancestors' rules bound each axis to [lo, hi]
            lo, hi = np.zeros(p, np.int64), inp.n_cuts.astype(np.int64).copy()
            q = h
            while q > 1:
                par_, right = q >> 1, q & 1
                a_ = axis[j, par_]
                if right:
                    lo[a_] = max(lo[a_], int(cut[j, par_]))
                else:
                    hi[a_] = min(hi[a_], int(cut[j, par_]) - 1)
                q = par_
            ok = np.flatnonzero(hi > lo)
            a = int(ok[rng.integers(ok.size)])
            axis[j, h] = a
            cut[j, h] = int(rng.integers(lo[a] + 1, hi[a] + 1))
        leaf[j, 1 << depth:2 << depth] = rng.normal(0.0, inp.hyper.sigma_mu, 1 << depth)
        hh = np.ones(n, np.int64)
        for _ in range(depth):
            a = axis[j, hh]
            right = inp.X_b[a, np.arange(n)] >= cut[j, hh]
            hh = 2 * hh + right
        idx[j] = hh
        f += leaf[j, hh].astype(np.float64)
    resid = (inp.y_c.astype(np.float64) - f).astype(np.float32)
    return dict(axis=axis, cut=cut, leaf=leaf, idx=idx, resid=resid,
                sigma2=inp.hyper.sigma2_init, sweep=0, next=0)


NO_CACHE = -1  # streamed residuals without an index cache


@pytest.mark.parametrize("residency", [REGS, STREAM, NO_CACHE])
@pytest.mark.parametrize("shape", ["d3_8_leaves", "d6_32_leaves", "d8_128_leaves"])
def test_lockstep_big_trees(shape, residency):
    """Trees far larger than the sampler grows by itself: 32 and 128 leaves
    take the LDS-bin reductions and mailboxes of up to 129 words; without an
    index cache, 31 internal nodes fill the 32-bit decision masks of the
    descent and 127 take the level-by-level descent.  8 leaves sit at the
    streamed pass's rank capacity (8 ranks a pass with the rank stash): a
    PRUNE's larger tree fills one pass with no spare slot, a GROW's 9 ranks
    take two passes, and a pruned tree's 7 leave the spare slot free."""
    kw = dict(idx_bytes=0) if residency == NO_CACHE else {}
    if shape == "d3_8_leaves":
        inp, depth = make_inputs(2, n=20011, p=12, m=12, **kw), 3
    elif shape == "d6_32_leaves":
        inp, depth = make_inputs(2, n=20011, p=12, m=12, **kw), 5
    else:
        inp, depth = make_inputs(5, n=30011, p=40, m=6, **kw), 7
    g = _gpu(inp, residency=STREAM if residency == NO_CACHE else residency)
    print(f"{shape}: grid={g.launch_info().grid} residency={g.launch_info().residency}",
          flush=True)
    g.set_state(_full_trees(inp, depth, np.random.default_rng(7)))
    rep = parity.lockstep(inp, g, seed=5, warm_sweeps=0, n_steps=2 * (inp.m + 1))
    print(f"  {rep}", flush=True)
    assert rep.moves > 0


@pytest.mark.parametrize("extra", [0, 1])
def test_register_residency_at_its_maximum(extra):
    """n = 256 workgroups x 512 threads x 8 chunks x 4 points fills every
    residual register of the grid (automatic residency keeps them on chip);
    one observation more streams them from HBM."""
    n = 256 * 512 * 8 * 4 + extra
    inp = make_inputs(2, n=n, p=10, m=6)
    g = _gpu(inp, launch=ORDINARY)
    info = g.launch_info()
    print(f"n={n}: grid={info.grid} chunks/thread={info.chunks_per_thread} "
          f"residency={info.residency}", flush=True)
    if info.grid < 256:
        pytest.skip("fewer than 256 compute units")
    if extra == 0:
        assert info.residency == REGS and info.chunks_per_thread == 8
    else:
        assert info.residency == STREAM and info.rank_stash == 1
    rep = parity.lockstep(inp, g, seed=inp.seed + 13, warm_sweeps=1, n_steps=inp.m + 1 + 3)
    print(f"  {rep}", flush=True)
    assert rep.moves > 0


@functools.lru_cache(maxsize=None)
def _stash_chunks():
    """Chunks of 4 points per thread the streamed kernel's LDS stash holds."""
    g = _gpu(make_inputs(2, n=1000, p=5, m=2), launch=ORDINARY, residency=STREAM)
    return g.launch_info().stash_chunks


@pytest.mark.parametrize("where", ["mixed", "full", "past"])
def test_streamed_at_the_stash_capacity(where):
    """One workgroup with 30 chunks of 4 points per thread (the stash in use,
    the residuals of the first few chunks in LDS and of the rest in HBM),
    with exactly as many chunks as the stash holds (every stash word in use)
    and with one more (the first size past it, a ragged last chunk): the
    kernel switches between its two passes there."""
    cap = _stash_chunks()
    cpt = {"mixed": 30, "full": cap, "past": cap + 1}[where]
    n = 2048 * cpt - (0 if where == "full" else 3)
    inp = make_inputs(4, n=n, p=12, m=16)
    g = _gpu(inp, grid=1, launch=ORDINARY, residency=STREAM)
    info = g.launch_info()
    print(f"{where}: n={n} chunks/thread={info.chunks_per_thread} rank_stash={info.rank_stash} "
          f"lds_resid_chunks={info.lds_resid_chunks}", flush=True)
    assert info.chunks_per_thread == cpt
    assert info.rank_stash == (0 if where == "past" else 1)
    if where == "mixed":
        assert 0 < info.lds_resid_chunks < cpt
    if where == "past":
        assert info.lds_resid_chunks == 0
    rep = parity.lockstep(inp, g, seed=inp.seed + 11, warm_sweeps=2, n_steps=inp.m + 1 + 9)
    print(f"  {rep}", flush=True)
    assert rep.moves > 0


@pytest.mark.parametrize("shape", ["u8", "u16", "d6_32_leaves", "no_index_cache"])
def test_streamed_without_the_rank_stash(shape):
    """More chunks per thread than the LDS rank stash holds (one workgroup,
    three chunks of 4 points per thread more than the stash, ragged): the
    streamed kernel reads each tree's rows again in the pass that applies it.
    Small trees, u8 and u16 caches, 32-leaf trees (two bin passes) and no
    index cache."""
    n = 2048 * (_stash_chunks() + 3) - 5
    if shape == "u16":
        inp = make_inputs(4, n=n, p=12, m=16)
    elif shape == "no_index_cache":
        inp = make_inputs(2, n=n, p=12, m=16, idx_bytes=0)
    else:
        inp = make_inputs(2, n=n, p=12, m=12 if shape == "d6_32_leaves" else 16)
    g = _gpu(inp, grid=1, launch=ORDINARY, residency=STREAM)
    info = g.launch_info()
    print(f"{shape}: grid={info.grid} chunks/thread={info.chunks_per_thread} "
          f"rank_stash={info.rank_stash}", flush=True)
    assert info.residency == STREAM and info.rank_stash == 0
    assert info.chunks_per_thread > info.stash_chunks
    if shape == "d6_32_leaves":
        g.set_state(_full_trees(inp, 5, np.random.default_rng(7)))
        rep = parity.lockstep(inp, g, seed=5, warm_sweeps=0, n_steps=2 * (inp.m + 1))
    else:
        rep = parity.lockstep(inp, g, seed=inp.seed + 3, warm_sweeps=2, n_steps=inp.m + 1 + 9)
    print(f"  {rep}", flush=True)
    assert rep.moves > 0


@pytest.mark.parametrize("residency", [REGS, STREAM])
def test_lockstep_exhausted_axes(residency):
    """Three predictors with three cuts each under depth-8 trees: paths run
    out of cuts on an axis within a few splits, so growable leaves, the axis
    pick (which skips exhausted axes) and the split probabilities of the
    children depend on the exhausted-axis count at every depth (the axes
    with cuts are fewer than the deepest path, so no shortcut applies)."""
    inp = make_inputs(5, n=20011, p=3, m=8)
    inp.X_b = (inp.X_b // 64).astype(np.uint8)  # 4 bins: cuts 1..3
    inp.n_cuts = np.full(inp.p, 3, np.int32)
    g = _gpu(inp, residency=residency)
    g.set_state(_full_trees(inp, 3, np.random.default_rng(11)))
    rep = parity.lockstep(inp, g, seed=9, warm_sweeps=0, n_steps=3 * (inp.m + 1))
    print(f"  {rep}", flush=True)
    assert rep.moves > 0


def test_lockstep_full_size_streamed():
    """Workload 4 (n = 1e7, u16 index cache): residuals streamed from HBM."""
    inp = _full(4)
    print(f"full workload 4: n={inp.n} p={inp.p} m={inp.m}", flush=True)
    g = _gpu(inp, launch=ORDINARY)
    assert g.launch_info().residency == STREAM
    g.step(20, inp.seed)
    assert g.status() == 0
    inv = parity.check_invariants(inp, g.get_state(), sweeps=20)
    print(f"  invariants after 20 untraced sweeps: {inv}", flush=True)
    rep = parity.lockstep(inp, g, seed=inp.seed, warm_sweeps=0, n_steps=inp.m + 1)
    print(f"  {rep}", flush=True)


# ---------------------------------------------------------------- several chains

@pytest.mark.parametrize("nchain,grid,residency,launch",
                         [(3, 0, REGS, COOP), (4, 5, REGS, ORDINARY), (3, 4, STREAM, COOP)])
def test_chains_lockstep(nchain, grid, residency, launch):
    inp = make_inputs(2, n=20011, p=30, m=30)
    print(f"chains={nchain} grid={grid} residency={residency} launch={launch}", flush=True)
    g = _gpu(inp, grid=grid, launch=launch, residency=residency, nchain=nchain)
    info = g.launch_info()
    assert info.nchain == nchain and info.residency == residency
    reps = parity.lockstep_chains(inp, g, seed=21, warm_sweeps=2, n_steps=31 * 2)
    for rep in reps:
        print(f"  {rep}", flush=True)
        assert rep.tree_steps > 0 and rep.moves > 0
    # different streams: the chains' trees differ
    states = [g.get_state(c) for c in range(nchain)]
    assert not np.array_equal(states[0]["leaf"], states[1]["leaf"])


@pytest.mark.parametrize("nchain,chunks,residency", [(2, 4, REGS), (4, 8, REGS), (16, 31, STREAM)])
def test_chains_full_size_lockstep(nchain, chunks, residency):
    """Workload 3 at full size with 2, 4 and 16 chains in the ordinary launch:
    2 and 4 chains keep their residuals in registers (4 and 8 chunks of 4
    points per thread); 16 chains of 16 workgroups stream them (31 chunks per
    thread, the first 4 in LDS): the shape bench.py's batched leg times.
    After untraced sweeps every chain's state meets the cache invariants, then
    every chain runs a whole sweep in lockstep with its oracle stream."""
    inp = _full(3)
    g = _gpu(inp, launch=ORDINARY, nchain=nchain)
    info = g.launch_info()
    print(f"workload 3, {nchain} chains: grid {info.grid} x {nchain}, {info.chunks_per_thread} "
          f"chunks per thread, residency {info.residency}", flush=True)
    assert info.nchain == nchain and info.chunks_per_thread == chunks
    assert info.residency == residency
    g.step(10, inp.seed)
    assert g.status() == 0
    for c in range(nchain):
        inv = parity.check_invariants(inp, g.get_state(c), sweeps=10, n_sample=64, seed=c)
        print(f"  chain {c} invariants: {inv}", flush=True)
    reps = parity.lockstep_chains(inp, g, seed=inp.seed, warm_sweeps=0, n_steps=inp.m + 1)
    for rep in reps:
        print(f"  {rep}", flush=True)
        assert rep.tree_steps == inp.m and rep.moves > 0


def test_chains_of_one_workgroup_lockstep():
    """Small n: every chain is one workgroup, whose mailbox words stay in LDS;
    six chains in lockstep with their oracle streams (ragged n: a partial
    last chunk of padding points)."""
    inp = make_inputs(1, n=997, p=8, m=20)
    g = _gpu(inp, launch=ORDINARY, nchain=6)
    info = g.launch_info()
    assert info.grid == 1 and info.nchain == 6
    reps = parity.lockstep_chains(inp, g, seed=13, warm_sweeps=3, n_steps=21 * 3)
    for rep in reps:
        print(f"  {rep}", flush=True)
        assert rep.tree_steps > 0 and rep.moves > 0


def test_chain0_equals_a_lone_chain():
    inp = make_inputs(2, n=30011, p=16, m=20)
    many = _gpu(inp, grid=6, nchain=5)
    one = _gpu(inp, grid=6)
    assert many.launch_info().chunks_per_thread == one.launch_info().chunks_per_thread
    many.step(4, 13)
    one.step(4, 13)
    sa, sb = many.get_state(0), one.get_state()
    for k in ["axis", "cut", "leaf", "idx", "resid"]:
        np.testing.assert_array_equal(sa[k], sb[k], err_msg=k)
    assert sa["sigma2"] == sb["sigma2"]
    assert many.status() == 0 and one.status() == 0


def test_chains_predict_and_set_state():
    inp = make_inputs(1, n=3001, p=10, m=30)
    g = _gpu(inp, nchain=3)
    g.step(4, 7)
    Xt = make_inputs(1, n=1999, p=10, m=30).X_b
    got = g.predict(Xt, inp.offset).cpu().numpy()
    assert got.shape == (3, 1999)
    for c in range(3):
        ch = parity.chain_from_state(inp, g.get_state(c), chain=c)
        np.testing.assert_array_equal(got[c], ch.predict(Xt, inp.offset))
    # set chain 1 to chain 2's state: from then on the two differ only by stream
    st2 = g.get_state(2)
    g.set_state(st2, chain=1)
    s1 = g.get_state(1)
    for k in ["axis", "cut", "leaf", "idx", "resid"]:
        np.testing.assert_array_equal(s1[k], st2[k], err_msg=k)
    assert s1["sigma2"] == st2["sigma2"]
    assert g.status() == 0


def test_move_statistics_count_every_step():
    """bart_move_stats against the per-step records of the same steps: runs
    that start and end inside a sweep, several launches, several chains."""
    inp = make_inputs(2, n=8009, p=20, m=25)
    g = _gpu(inp, nchain=2, launch=ORDINARY)
    g.step(3, 17)
    before = [g.move_stats(c) for c in range(2)]
    assert all(b["tree_steps"] == 3 * inp.m for b in before)
    n_steps = 2 * (inp.m + 1) + 7
    tr = g.debug_steps(n_steps, 17)                    # ends inside a sweep
    tr2 = g.debug_steps(inp.m + 1, 17)                 # starts inside one
    for c in range(2):
        recs = np.concatenate([tr[c], tr2[c]])
        t = recs[recs["kind"] == 0]
        after = g.move_stats(c)
        d = {k: after[k] - before[c][k] for k in after}
        assert d["tree_steps"] == len(t)
        assert d["grow_proposed"] == int((t["move"] == 1).sum())
        assert d["prune_proposed"] == int((t["move"] == 2).sum())
        assert d["grow_accepted"] == int(((t["move"] == 1) & (t["accept"] == 1)).sum())
        assert d["prune_accepted"] == int(((t["move"] == 2) & (t["accept"] == 1)).sum())
        merged = ((t["move"] == 1) & (t["accept"] == 0)) | ((t["move"] == 2) & (t["accept"] == 1))
        assert d["leaves"] == int((t["n_leaves"] - merged).sum())
    assert g.status() == 0


# ---------------------------------------------------------------- probit

@pytest.mark.parametrize("residency,nchain", [(REGS, 1), (STREAM, 1), (REGS, 2)])
def test_probit_lockstep(residency, nchain):
    """Binary y: tree steps as in regression (sigma^2 = 1), and the step that
    ends a sweep draws the latents; two whole sweeps in lockstep."""
    from paper_2410_23244_amd.inputs import make_probit_inputs

    inp = make_probit_inputs(n=20011, p=10, m=30)
    print(f"probit residency={residency} nchain={nchain}", flush=True)
    g = _gpu(inp, residency=residency, nchain=nchain)
    assert g.launch_info().residency == residency
    st = g.get_state()
    ybin = inp.y_c > 0
    assert ((st["latent"] > 0) == ybin).all() and st["sigma2"] == 1.0
    reps = parity.lockstep_chains(inp, g, seed=31, warm_sweeps=3, n_steps=2 * (inp.m + 1))
    for c, rep in enumerate(reps):
        print(f"  {rep}", flush=True)
        assert rep.tree_steps > 0 and rep.moves > 0
        s = g.get_state(c)
        assert s["sigma2"] == 1.0 and ((s["latent"] > 0) == ybin).all()


def test_probit_recovers_class_probabilities():
    from scipy import stats

    from paper_2410_23244_amd.inputs import column, make_probit_inputs

    inp = make_probit_inputs(n=50000, p=10, m=50)
    g = _gpu(inp, nchain=2)
    g.step(100, 3)
    cols = [column(2, a, inp.n).astype(np.float64) for a in range(4)]
    gtrue = (1.5 * np.sin(2 * np.pi * cols[0]) + 2.0 * (cols[1] - 0.5) + cols[2] * cols[3]
             - 0.25)
    prob = np.zeros(inp.n)
    for _ in range(50):
        g.step(1, 3)
        f = g.predict(inp.X_b, inp.offset).cpu().numpy().astype(np.float64)
        prob += stats.norm.cdf(f).mean(axis=0)
    prob /= 50
    err = np.abs(prob - stats.norm.cdf(gtrue)).mean()
    print(f"probit mean |p - p_true| = {err:.4f}", flush=True)
    assert err < 0.05
    assert g.status() == 0


# ---------------------------------------------------------------- no index cache

@pytest.mark.parametrize("cfg,over", [(2, dict(n=40003, p=30, m=40)),
                                      (5, dict(n=25003, p=1000, m=120)),
                                      (1, dict(n=301, p=3, m=4, D=2)),
                                      (5, dict(n=20011, p=50, m=40, D=7))])
def test_no_index_cache_lockstep(cfg, over):
    """idx_bytes = 0: the trees route the observations by Algorithm 1 every
    step; lockstep against the oracle, whose cache the device exports.  Depth
    2 and 6 take the decision bits by heap slot, depth 7 and 8 by the node's
    place in the list of internal nodes."""
    inp = make_inputs(cfg, **over, idx_bytes=0)
    g = _gpu(inp, grid=4, launch=ORDINARY)
    assert g.launch_info().residency == STREAM
    rep = parity.lockstep(inp, g, seed=inp.seed + 7, warm_sweeps=2, n_steps=inp.m + 1 + 9)
    print(f"  {rep}", flush=True)
    assert rep.tree_steps > 0 and rep.moves > 0


def test_no_index_cache_equals_the_cached_kernel():
    """Same partition, same sums: the chain without an index cache is the
    chain with one, bit for bit, across launches that split sweeps."""
    inp8 = make_inputs(2, n=30011, p=16, m=25)
    inp0 = make_inputs(2, n=30011, p=16, m=25, idx_bytes=0)
    a = _gpu(inp8, grid=5, residency=STREAM, nchain=2)
    b = _gpu(inp0, grid=5, nchain=2)
    for k in (3, 1, 2):
        a.step(k, 29)
        b.step(k, 29)
    a.debug_steps(13, 29)
    b.debug_steps(13, 29)
    for c in range(2):
        sa, sb = a.get_state(c), b.get_state(c)
        for key in ["axis", "cut", "leaf", "idx", "resid"]:
            np.testing.assert_array_equal(sa[key], sb[key], err_msg=key)
        assert sa["sigma2"] == sb["sigma2"]
    # a state loaded into a chain without a cache continues identically
    st = a.get_state(0)
    c0 = _gpu(inp0, grid=5)
    c8 = _gpu(inp8, grid=5, residency=STREAM)
    c0.set_state(st)
    c8.set_state(st)
    c0.debug_steps(20, 5)
    c8.debug_steps(20, 5)
    s0, s8 = c0.get_state(), c8.get_state()
    for key in ["axis", "cut", "leaf", "idx", "resid"]:
        np.testing.assert_array_equal(s0[key], s8[key], err_msg=key)
    assert a.status() == 0 and b.status() == 0 and c0.status() == 0
