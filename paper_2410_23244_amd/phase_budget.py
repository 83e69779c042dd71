"""Per-phase time budget of a tree step of the register sweep kernel, from
the diagnostic build libbart_clocks.so (build.build(clocks=True)).

Thread 0 of every workgroup stamps the wall clock (100 MHz) at the phase
boundaries of 64 consecutive tree steps of one launch, and every workgroup
counts the mailbox loads its polls issue.  Phases of a tree step j:
  route      route of tree j+1 (rank of every point in its larger tree)
  prefetch   loads of later trees' rows and decision data, rank table of
             tree j+2, tree j's count-only constants
  gather     polls of every workgroup's partial sums of tree j
  decide     MH decision and leaf draws (wave 0: the decision)
  barrier    until every wave has its part of the decision
  update     residual update and index-row rewrite
  finish     the owner's write of tree j
  reduce     partial sums of tree j+1 and their post (split into the bin
             updates, the bin barrier, rank 0's cross-wave total and post,
             and the rest)
The script prints medians over workgroups and steps, the step period, the
spread of the posts and the time from the last post to the first and last
completed gathers, and the mailbox loads per step against G^2 (L + 1).

  python -m paper_2410_23244_amd.phase_budget --config 3 [--out clocks.npy]

Runs on cuda:0; not part of the product path (a diagnostic build)."""
from __future__ import annotations

import argparse
import ctypes as C
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))

K_GRID, K_STEPS, K_PH = 256, 48, 20  # kMaxGrid, kClockSteps, kClockPh
K_START = 205                        # kClockStart
K_SPH = 9                            # kSigmaPh
PHASES = ["route", "prefetch", "gather", "decide", "barrier", "update", "finish", "reduce"]
# stamps 9-11 (inside the reduce: bins done, bin barrier passed, rank 0 posted)
SUB = ["bins", "bin barrier", "rank-0 total and post", "rest of reduce"]


def run(config: int, warmup: int, seed: int, out: str | None) -> dict:
    import torch

    from paper_2410_23244_amd import bart as B
    from paper_2410_23244_amd.build import CLOCKS_LIB
    from paper_2410_23244_amd.inputs import make_inputs

    if not os.path.exists(CLOCKS_LIB):
        raise RuntimeError(f"{CLOCKS_LIB} is missing: build it with build.build(clocks=True)")
    B.LIB_PATH = CLOCKS_LIB
    lib = B.lib()
    lib.bart_phase_clocks.argtypes = [C.c_void_p, C.c_size_t]
    lib.bart_phase_clocks.restype = C.c_int
    inp = make_inputs(config)
    g = B.from_inputs(inp, launch=B.BART_LAUNCH_ORDINARY)
    info = g.launch_info()
    if info.residency != B.BART_RESID_REGISTERS or info.nchain != 1:
        raise RuntimeError("the phase clocks cover the register kernel of one chain")
    G = info.grid
    g.step(warmup, seed)
    sweeps = -(-(K_START + K_STEPS) // (inp.m + 1))  # one launch covering the window
    g.step(sweeps, seed)
    torch.cuda.synchronize()
    buf = np.zeros(K_GRID * K_STEPS * K_PH, np.uint64)
    if lib.bart_phase_clocks(buf.ctypes.data, buf.size) != 0:
        raise RuntimeError(lib.bart_last_error().decode())
    ts = buf.reshape(K_GRID, K_STEPS, K_PH).astype(np.int64)[:G]
    if out:
        np.save(out, ts)
    loads = ts[:, :, K_PH - 1]
    clk = ts[:, :, : K_PH - 1] * 10  # ns
    sub = clk[:, :, [7, 9, 10, 11, 8]]  # finish, bins, barrier, rank-0 post, end
    ok = (clk[:, :, 0] > 0).all(0) & (clk[:, :, 8] > 0).all(0)  # tree steps (not sigma^2)
    clk, loads, sub = clk[:, ok], loads[:, ok], sub[:, ok]
    d = np.diff(clk[:, :, :9], axis=2)
    ds = np.diff(sub, axis=2)
    res = {"config": config, "workload": inp.workload, "grid": G, "tree_steps": int(ok.sum()),
           "first_step": K_START,
           "phase_median_ns": {p: float(np.median(d[:, :, k])) for k, p in enumerate(PHASES)},
           "phase_p90_ns": {p: float(np.percentile(d[:, :, k], 90)) for k, p in enumerate(PHASES)},
           "reduce_parts_median_ns": {p: float(np.median(ds[:, :, k])) for k, p in enumerate(SUB)}}
    post, gd = clk[:, :, 8], clk[:, :, 3]
    res["step_period_median_ns"] = float(np.median(np.diff(clk[0, :, 0])))
    res["post_spread_median_ns"] = float(np.median(post.max(0) - post.min(0)))
    last = post[:, :-1].max(0)
    rel = gd[:, 1:] - last
    res["last_post_to_first_gather_done_median_ns"] = float(np.median(rel.min(0)))
    res["last_post_to_last_gather_done_median_ns"] = float(np.median(rel.max(0)))
    res["gathered_to_posted_median_ns"] = float(np.median(post - gd))
    lw = post.argmax(0)
    res["last_poster_xcd_histogram (wg mod 8)"] = np.bincount(lw % 8, minlength=8).tolist()
    # the last thread (a polling thread): its reduce ends (stamp 12) one step
    # before the loop top (13), its route (14), decision-data and row loads
    # (15, 16), poll start (17) and poll end (18)
    pol = [clk[:, :-1, 12]] + [clk[:, 1:, q] for q in range(13, 19)]
    names = ["reduce end to loop top", "route", "decision-data loads", "row loads",
             "to polls start", "polls"]
    lastpost = post[:, :-1].max(0)
    res["poller_median_ns"] = {nm: float(np.median(pol[i + 1] - pol[i])) for i, nm in enumerate(names)}
    res["poller_median_ns"]["polls start after last post"] = float(np.median(pol[5] - lastpost))
    res["poller_median_ns"]["polls end after last post"] = float(np.median(pol[6] - lastpost))
    late, cols = lw[:-1], np.arange(len(lw) - 1)
    res["poller_last_poster_median_ns"] = {
        nm: float(np.median((pol[i + 1] - pol[i])[late, cols])) for i, nm in enumerate(names)}
    # mailbox loads: words of every mailbox once, G^2 (L+1) per step, plus re-polls
    res["mailbox_loads_per_step_median"] = float(np.median(loads.sum(0)))
    res["mailbox_loads_per_wg_step_median"] = float(np.median(loads))
    res["mailbox_loads_per_wg_step_min"] = float(loads.min())
    # the last sigma^2 step of the launch
    lib.bart_sigma_clocks.argtypes = [C.c_void_p, C.c_size_t]
    lib.bart_sigma_clocks.restype = C.c_int
    sb = np.zeros(K_GRID * K_SPH, np.uint64)
    if lib.bart_sigma_clocks(sb.ctypes.data, sb.size) != 0:
        raise RuntimeError(lib.bart_last_error().decode())
    sc = sb.reshape(K_GRID, K_SPH).astype(np.int64)[:G] * 10
    ds = np.diff(sc, axis=1)
    names = ["sums of squares", "proposals (owner wave 0)", "leaf normals", "barrier",
             "release (wave 0)", "gather of the sums", "draw", "refill of the next sweep"]
    res["sigma2_step_median_ns"] = {nm: float(np.median(ds[:, k])) for k, nm in enumerate(names)}
    res["sigma2_step_total_median_ns"] = float(np.median(sc[:, K_SPH - 1] - sc[:, 0]))
    owners = min(G, inp.m)
    res["proposal_owner_max_ns"] = float(ds[:owners, 1].max())
    g.close()
    return res


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--seed", type=int, default=3)
    ap.add_argument("--out", default=None, help="save the raw clocks (.npy)")
    a = ap.parse_args()
    print(json.dumps(run(a.config, a.warmup, a.seed, a.out), indent=1), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
