"""Benchmark of the BART sweep on one MI355X.

A step is one full MCMC sweep (every tree updated in order, then sigma^2)
over the synthetic workload n=1e6, p=100, ntree=200, depth 6, uint8 index
cache.  Inputs are generated and uploaded before the timed region; the timed
region is one bart_step(K) launch, bracketed by device synchronisations and
timed with HIP events on the chain's stream.  Prints one JSON line.

Roofline: the algorithmic bytes of a tree step are (9 + 2 s_idx) per
observation (read the index row and the predictor row, read and write the
residual, write the index row) plus 4 bytes per observation per sweep for
sigma^2; achieved = algorithmic bytes / launch duration, against 8 TB/s.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("full MCMC sweeps/sec (all trees) at n=1e6,p=100,ntree=200; achieved HBM GB/s")
HBM_PEAK_GBS = 8000.0


def model_bytes_per_sweep(n: int, m: int, idx_bytes: int) -> int:
    return m * n * (9 + 2 * idx_bytes) + 4 * n


def cpu_baseline(inp, state, seed: int, sweeps: int) -> dict:
    """The oracle, single-threaded, on the host, from the device chain's state."""
    import oracle
    from tests.parity import chain_from_state

    ch = chain_from_state(inp, state)
    t = time.perf_counter()
    ch.sweeps(seed, sweeps)
    dt = time.perf_counter() - t
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
                      f"after warm-up, {dt:.1f} s on 1 thread of {cpu} "
                      f"(host has {os.cpu_count()} logical CPUs)"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000, help="timed sweeps")
    ap.add_argument("--warmup", type=int, default=10, help="untimed sweeps")
    ap.add_argument("--config", type=int, default=3, help="workload number (3 = headline)")
    ap.add_argument("--cpu-sweeps", type=int, default=5, help="oracle sweeps (0 = skip)")
    ap.add_argument("--seed", type=int, default=3)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the sweep is built and measured on a single MI355X)", file=sys.stderr)
        return 2

    import torch

    from paper_2410_23244_amd.bart import from_inputs
    from paper_2410_23244_amd.inputs import make_inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    inp = make_inputs(args.config)
    print(f"[bench] inputs {inp.workload} in {time.perf_counter() - t0:.1f} s", file=sys.stderr,
          flush=True)
    g = from_inputs(inp)
    info = g.launch_info()
    stream = g.stream
    if args.warmup:
        g.step(args.warmup, args.seed)
    torch.cuda.synchronize()
    assert g.status() == 0, "device error during warm-up"
    print(f"[bench] warm-up {args.warmup} sweeps done", file=sys.stderr, flush=True)

    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    e0.record(stream)
    g.step(args.steps, args.seed)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = e0.elapsed_time(e1)
    assert g.status() == 0, "device error during the timed sweeps"
    sec = ms / 1e3
    sweeps_per_s = args.steps / sec
    per_sweep = model_bytes_per_sweep(inp.n, inp.m, inp.idx_bytes)
    achieved = per_sweep * args.steps / sec / 1e9
    print(f"[bench] {args.steps} sweeps: events {ms:.1f} ms, wall {wall * 1e3:.1f} ms",
          file=sys.stderr, flush=True)

    cpu = None
    if args.cpu_sweeps > 0:
        st = g.get_state()
        cpu = cpu_baseline(inp, st, args.seed, args.cpu_sweeps)
        print(f"[bench] oracle {cpu['value']:.3f} sweeps/s", file=sys.stderr, flush=True)

    line = {
        "metric": METRIC,
        "value": sweeps_per_s,
        "unit": "sweeps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": inp.workload, "n": inp.n, "p": inp.p, "ntree": inp.m,
                   "max_depth": inp.D, "idx_bytes": inp.idx_bytes,
                   "sweeps_per_launch": args.steps, "grid": info.grid,
                   "chunks_per_thread": info.chunks_per_thread, "parallelism": "1 GPU"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None},
        "cpu_baseline": cpu,
        "host": platform.node(),
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
