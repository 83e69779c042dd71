"""Benchmark of the BART sweep on one MI355X.

A step is one full MCMC sweep (every tree updated in order, then sigma^2)
over the synthetic workload n=1e6, p=100, ntree=200, depth 6, uint8 index
cache.  Inputs are generated and uploaded before the timed region.  Warm-up
and timed sweeps run as bart_step calls of --sweeps-per-launch sweeps each
(one kernel launch per call), the remainder as one shorter call, so any
--steps >= 1 and --warmup >= 0 run; each timed launch is bracketed by HIP
events on the chain's stream, and the whole timed region by device
synchronisations.  Prints one JSON line.

--chains C runs C independent chains in the same launches (multi-chain
batching); value is then the chain-sweeps per second summed over the chains
and the roofline counts every chain's bytes.  The single-chain headline run
also times 16 chains batched on the same workload after its own measurement
and reports them in a separate 'batched' object (--batched sets the count,
0 turns it off); value stays the single chain's.

Roofline: the algorithmic bytes of a tree step are (9 + 2 s_idx) per
observation (read the index row and the predictor row, read and write the
residual, write the index row) plus 4 bytes per observation per sweep for
sigma^2; achieved = algorithmic bytes per launch / average launch duration,
against 8 TB/s.  traffic = HBM bytes per launch measured by the FETCH_SIZE
and WRITE_SIZE counters (calibrated on a plain copy) for the current kernel
sources, else null; measured_hbm_gbs = traffic / average launch duration.
copy_ceiling = the bandwidth of a plain 1 GiB device copy timed in the same
run, the ceiling a streaming kernel can reach on this GPU.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("full MCMC sweeps/sec (all trees) at n=1e6,p=100,ntree=200; achieved HBM GB/s")
HBM_PEAK_GBS = 8000.0


def model_bytes_per_sweep(n: int, m: int, idx_bytes: int) -> int:
    return m * n * (9 + 2 * idx_bytes) + 4 * n


def launch_plan(sweeps: int, per_launch: int) -> list:
    """Sweeps of each bart_step call (one kernel launch each) that together run
    `sweeps` sweeps: full launches of per_launch, then one shorter launch for
    the remainder.  Any sweeps >= 0 and per_launch >= 1 are accepted."""
    if sweeps < 0 or per_launch < 1:
        raise ValueError("sweeps must be >= 0 and per_launch >= 1")
    plan = [per_launch] * (sweeps // per_launch)
    if sweeps % per_launch:
        plan.append(sweeps % per_launch)
    return plan


def cpu_baseline(inp, state, seed: int, sweeps: int) -> dict:
    """The oracle, single-threaded and pinned to one host core, on the host,
    from the device chain's state."""
    import oracle

    ch = oracle.chain_from_state(inp, state)
    prev = os.sched_getaffinity(0) if hasattr(os, "sched_getaffinity") else None
    core = min(prev) if prev else None
    if core is not None:
        os.sched_setaffinity(0, {core})
    try:
        t = time.perf_counter()
        ch.sweeps(seed, sweeps)
        dt = time.perf_counter() - t
    finally:
        if prev is not None:
            os.sched_setaffinity(0, prev)
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    del oracle
    return {"value": sweeps / dt, "unit": "sweeps/s", "cores": 1, "kind": "oracle",
            "sample": f"{sweeps} sweeps of the same workload from the device chain's state "
                      f"after the timed sweeps, {dt:.1f} s on 1 thread pinned to core {core} "
                      f"of {cpu} (host has {os.cpu_count()} logical CPUs)"}


def copy_probe(mib: int) -> int:
    """A plain elementwise copy (dst = -src) of known size for counter calibration."""
    import torch

    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": 4 * n, "copy_probe_bytes_written": 4 * n,
                      "launches": 3}), flush=True)
    return 0


def copy_ceiling_gbs(mib: int = 1024, reps: int = 5) -> float:
    """HBM bandwidth a plain device copy sustains on this GPU: read + write
    bytes of a 1 GiB f32 copy over its HIP-event time (best of reps)."""
    import torch

    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    best = float("inf")
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del src, dst
    torch.cuda.empty_cache()
    return 2 * 4 * n / (best / 1e3) / 1e9


SWEEP_SOURCES = ("common.hpp", "propose.hpp", "rng.hpp", "sweep.hpp")


def kernel_source_digest() -> str:
    """sha256 over the sources of the sweep kernels (to tell whether stored
    counters are stale); host code and the predict kernel do not enter."""
    import hashlib

    d = os.path.join(ROOT, "paper_2410_23244_amd", "csrc")
    h = hashlib.sha256()
    for name in SWEEP_SOURCES:
        with open(os.path.join(d, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def stored_traffic(workload: str, sweeps_per_launch: int):
    """HBM bytes per launch from the committed counter summary, or None when it was
    taken on other sources or another workload."""
    path = os.path.join(ROOT, "profiles", "sweep_kernel_traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_src_sha256") != kernel_source_digest():
        return None
    for r in rec.get("records", []):
        if r.get("workload") == workload:
            return (r["fetch_bytes_per_sweep"] + r["write_bytes_per_sweep"]) * sweeps_per_launch
    return None


def bench_predict(args, inp, g) -> int:
    """Time bart_predict of the warmed-up chains on NT points of the same generator."""
    import torch

    from paper_2410_23244_amd.inputs import make_inputs

    nt = args.predict
    Xt = make_inputs(args.config, n=nt).X_b
    Xd, _ = g.upload_x(Xt)
    out = torch.empty((args.chains, nt), dtype=torch.float32, device=g.device)
    from paper_2410_23244_amd.bart import bart_predict

    def once():
        bart_predict(g.h, Xd.data_ptr(), Xd.shape[1], nt, inp.offset, out.data_ptr())

    for _ in range(3):
        once()
    torch.cuda.synchronize()
    reps = max(1, args.steps // 100)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(g.stream)
    for _ in range(reps):
        once()
    e1.record(g.stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    trav = args.chains * nt * inp.m
    line = {"metric": f"sum-of-trees predictions/sec at n_t={nt}, ntree={inp.m}, D={inp.D}, "
                      f"p={inp.p}",
            "value": args.chains * nt / (ms / 1e3), "unit": "points/s", "n_gpus": 1,
            "steps": reps, "warmup": 3, "ms_per_step": ms, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "f64 sum, u8 route",
            "data": "synthetic", "tree_traversals_per_s": trav / (ms / 1e3),
            "config": {"workload": f"bart_predict_nt{nt}_" + inp.workload, "nchain": args.chains,
                       "trees_after_warmup_sweeps": args.warmup}}
    print(json.dumps(line), flush=True)
    return 0


def make_parser() -> argparse.ArgumentParser:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000, help="timed sweeps")
    ap.add_argument("--warmup", type=int, default=100, help="untimed sweeps before timing")
    ap.add_argument("--sweeps-per-launch", type=int, default=100,
                    help="sweeps per bart_step call (one kernel launch each)")
    ap.add_argument("--launch", choices=["ordinary", "cooperative"], default="ordinary",
                    help="how the sweep kernel is launched (kernel tracers cannot record "
                         "cooperative launches)")
    ap.add_argument("--config", type=int, default=3, help="workload number (3 = headline)")
    ap.add_argument("--cpu-sweeps", type=int, default=20, help="oracle sweeps (0 = skip)")
    ap.add_argument("--seed", type=int, default=3)
    ap.add_argument("--chains", type=int, default=1, help="independent chains per launch")
    ap.add_argument("--batched", type=int, default=-1, metavar="C",
                    help="after the main line's measurement, also time C chains batched in the "
                         "same launches on the same workload and report them under 'batched' "
                         "(-1: 16 for the single-chain headline workload, else off; 0: off)")
    ap.add_argument("--grid", type=int, default=0, help="workgroups per chain (0 = automatic)")
    ap.add_argument("--no-index-cache", action="store_true",
                    help="run without the [ntree][n] index cache (Algorithm 1 every tree step)")
    ap.add_argument("--predict", type=int, default=0, metavar="NT",
                    help="after the warm-up, time bart_predict on NT points instead of sweeps")
    ap.add_argument("--no-copy-ceiling", dest="copy_ceiling", action="store_false",
                    help="skip the timed plain copy that gives roofline.copy_ceiling")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (read MIB, write MIB) three "
                         "times, to calibrate HBM byte counters, and exit")
    return ap


def plans(args) -> tuple:
    """Sweeps per warm-up launch and per timed launch; ValueError on bad sizes."""
    if args.steps < 1 or args.warmup < 0 or args.sweeps_per_launch < 1:
        raise ValueError("--steps and --sweeps-per-launch must be >= 1, --warmup >= 0")
    return (launch_plan(args.warmup, args.sweeps_per_launch),
            launch_plan(args.steps, args.sweeps_per_launch))


def main() -> int:
    args = make_parser().parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the sweep is built and measured on a single MI355X)", file=sys.stderr)
        return 2
    S = args.sweeps_per_launch
    try:
        warm_plan, plan = plans(args)
    except ValueError as e:
        print(str(e), file=sys.stderr)
        return 2

    import torch

    from paper_2410_23244_amd.bart import (BART_LAUNCH_COOPERATIVE, BART_LAUNCH_ORDINARY,
                                           from_inputs)
    from paper_2410_23244_amd.inputs import make_inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_probe:
        return copy_probe(args.copy_probe)
    t0 = time.perf_counter()
    inp = make_inputs(args.config, idx_bytes=0 if args.no_index_cache else None)
    print(f"[bench] inputs {inp.workload} in {time.perf_counter() - t0:.1f} s", file=sys.stderr,
          flush=True)
    mode = BART_LAUNCH_ORDINARY if args.launch == "ordinary" else BART_LAUNCH_COOPERATIVE
    C = args.chains
    g = from_inputs(inp, launch=mode, nchain=C, grid=args.grid)
    info = g.launch_info()
    kernel = (f"bart::sweep_kernel_stream<{max(1, inp.idx_bytes)}, "
              f"{'true' if inp.idx_bytes == 0 else 'false'}, "
              f"{'true' if info.rank_stash else 'false'}>" if info.residency == 2 else
              f"bart::sweep_kernel<{info.chunks_per_thread}, {inp.idx_bytes}>")
    stream = g.stream
    for k in warm_plan:
        g.step(k, args.seed)
    torch.cuda.synchronize()
    assert g.status() == 0, "device error during warm-up"
    print(f"[bench] warm-up {args.warmup} sweeps done in {len(warm_plan)} launches",
          file=sys.stderr, flush=True)
    if args.predict:
        return bench_predict(args, inp, g)

    L = len(plan)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * L)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for i, k in enumerate(plan):
        ev[2 * i].record(stream)
        g.step(k, args.seed)
        ev[2 * i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    assert g.status() == 0, "device error during the timed sweeps"
    ms = ev[0].elapsed_time(ev[-1])
    launch_ms = [ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(L)]
    avg_launch = sum(launch_ms) / L
    sweeps_per_launch = args.steps / L  # mean over the timed launches
    sweeps_per_s = C * args.steps / (ms / 1e3)
    # without an index cache the same model bytes as the u8 cache are counted
    per_sweep = C * model_bytes_per_sweep(inp.n, inp.m, max(1, inp.idx_bytes))
    achieved = per_sweep * sweeps_per_launch / (avg_launch / 1e3) / 1e9
    print(f"[bench] {args.steps} sweeps in {L} launches {plan}: events {ms:.2f} ms, wall "
          f"{wall * 1e3:.1f} ms, per launch {min(launch_ms):.3f}..{max(launch_ms):.3f} ms",
          file=sys.stderr, flush=True)
    copy_gbs = copy_ceiling_gbs() if args.copy_ceiling else None

    cpu = None
    if args.cpu_sweeps > 0:
        st = g.get_state()
        cpu = cpu_baseline(inp, st, args.seed, args.cpu_sweeps)
        print(f"[bench] oracle {cpu['value']:.3f} sweeps/s", file=sys.stderr, flush=True)

    batched = None
    nb = args.batched if args.batched >= 0 else (
        16 if args.config == 3 and C == 1 and args.grid == 0 and not args.no_index_cache else 0)
    if nb > 1:
        # the same workload with nb chains in the same launches: chain-sweeps
        # per second summed over the chains, timed like the main line
        gb = from_inputs(inp, launch=mode, nchain=nb)
        ib = gb.launch_info()
        for k in warm_plan:
            gb.step(k, args.seed)
        torch.cuda.synchronize()
        planb = launch_plan(max(1, args.steps // 2), S)
        Lb = len(planb)
        evb = [torch.cuda.Event(enable_timing=True) for _ in range(2 * Lb)]
        for i, k in enumerate(planb):
            evb[2 * i].record(gb.stream)
            gb.step(k, args.seed)
            evb[2 * i + 1].record(gb.stream)
        torch.cuda.synchronize()
        assert gb.status() == 0, "device error during the batched sweeps"
        msb = evb[0].elapsed_time(evb[-1])
        sweeps_b = sum(planb)
        achb = (nb * model_bytes_per_sweep(inp.n, inp.m, max(1, inp.idx_bytes)) * sweeps_b /
                (sum(evb[2 * i].elapsed_time(evb[2 * i + 1]) for i in range(Lb)) / 1e3) / 1e9)
        batched = {"chains": nb, "value": nb * sweeps_b / (msb / 1e3), "unit": "chain-sweeps/s",
                   "steps": sweeps_b, "ms_per_step": msb / sweeps_b, "grid_per_chain": ib.grid,
                   "chunks_per_thread": ib.chunks_per_thread,
                   "residency": "streamed" if ib.residency == 2 else "registers",
                   "lds_resid_chunks": ib.lds_resid_chunks,
                   "roofline_achieved_gbs": achb, "roofline_frac": achb / HBM_PEAK_GBS}
        print(f"[bench] {nb} chains batched: {batched['value']:.1f} chain-sweeps/s",
              file=sys.stderr, flush=True)
        gb.close()

    traffic = (stored_traffic(inp.workload, sweeps_per_launch)
               if C == 1 and not args.no_index_cache else None)
    roofline = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS, "traffic": traffic, "kernel": kernel,
                "avg_launch_ms": avg_launch, "sweeps_per_launch": sweeps_per_launch,
                "algorithmic_bytes_per_launch": per_sweep * sweeps_per_launch,
                # HBM bytes the counters measured per launch over the launch time: with
                # residuals in registers the kernel moves far fewer bytes than the
                # algorithmic count and is bound by the latency of its per-tree steps
                "measured_hbm_gbs": traffic / (avg_launch / 1e3) / 1e9 if traffic else None,
                "limiter": ("per-tree-step latency (grid exchange and decision); residuals "
                            "stay in registers" if info.residency != 2 else
                            "HBM bandwidth and the latency of the fused per-tree pass")}
    if traffic:
        roofline["measured_hbm_frac"] = roofline["measured_hbm_gbs"] / HBM_PEAK_GBS
    if copy_gbs:
        roofline["copy_ceiling"] = {"gbs": copy_gbs, "frac_of_peak": copy_gbs / HBM_PEAK_GBS,
                                    "achieved_frac_of_copy": achieved / copy_gbs,
                                    "kernel": "device-to-device copy of 1 GiB (f32), "
                                              "read + write bytes over its event time"}
    metric = METRIC
    if args.config != 3 or C > 1 or args.no_index_cache:
        metric = (f"full MCMC sweeps/sec (all trees) at n={inp.n},p={inp.p},ntree={inp.m},"
                  f"D={inp.D}" + (f", summed over {C} chains" if C > 1 else "") +
                  (", no index cache" if args.no_index_cache else "") +
                  "; achieved HBM GB/s")
    line = {
        "metric": metric,
        "value": sweeps_per_s,
        "unit": "sweeps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "launches": plan,
        "ms_per_step": ms / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": inp.workload, "n": inp.n, "p": inp.p, "ntree": inp.m,
                   "max_depth": inp.D, "idx_bytes": inp.idx_bytes, "sweeps_per_launch": S,
                   "launch": args.launch, "grid": info.grid, "nchain": C,
                   "residency": "streamed" if info.residency == 2 else "registers",
                   "chunks_per_thread": info.chunks_per_thread, "parallelism": "1 GPU"},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if batched is not None:
        line["batched"] = batched
    print(json.dumps(line), flush=True)
    g.close()
    torch.cuda.synchronize()
    return 0


if __name__ == "__main__":
    sys.exit(main())
