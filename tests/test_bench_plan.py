"""Host logic of bench.py: its argument parser and launch plan accept the
driver's command line, and stored counter bytes are used only for the sources
they were taken on (no GPU needed)."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

import bench


def _plans(argv):
    return bench.plans(bench.make_parser().parse_args(argv))


def test_driver_command_gives_a_valid_plan():
    warm, timed = _plans(["--gpus", "1", "--steps", "20", "--warmup", "5"])
    assert warm == [5] and timed == [20]


def test_default_plan():
    warm, timed = _plans([])
    assert warm == [100] and timed == [100] * 10


def test_remainder_launch():
    warm, timed = _plans(["--steps", "250", "--warmup", "0", "--sweeps-per-launch", "100"])
    assert warm == [] and timed == [100, 100, 50]


@pytest.mark.parametrize("sweeps,per", [(0, 7), (1, 100), (250, 100), (300, 100), (7, 3)])
def test_plan_sums_and_bounds(sweeps, per):
    plan = bench.launch_plan(sweeps, per)
    assert sum(plan) == sweeps
    assert all(1 <= k <= per for k in plan)
    assert plan == sorted(plan, reverse=True)


@pytest.mark.parametrize("argv", [["--steps", "0"], ["--warmup", "-1"],
                                  ["--sweeps-per-launch", "0"]])
def test_plan_rejects_bad_sizes(argv):
    with pytest.raises(ValueError):
        _plans(argv)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_stored_traffic_follows_the_kernel_sources(tmp_path, monkeypatch):
    """The counter bytes in profiles/ enter the bench line only for their own
    workload and only while the sweep-kernel sources hash to the digest
    recorded with them."""
    import json
    import shutil

    src = os.path.join(bench.ROOT, "paper_2410_23244_amd", "csrc")
    dst = tmp_path / "paper_2410_23244_amd" / "csrc"
    dst.mkdir(parents=True)
    for name in bench.SWEEP_SOURCES:
        shutil.copy(os.path.join(src, name), dst / name)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (tmp_path / "profiles").mkdir()
    rec = {"kernel_src_sha256": bench.kernel_source_digest(),
           "records": [{"workload": "w", "fetch_bytes_per_sweep": 300, "write_bytes_per_sweep": 100}]}
    (tmp_path / "profiles" / "sweep_kernel_traffic.json").write_text(json.dumps(rec))
    assert bench.stored_traffic("w", 10) == 4000
    assert bench.stored_traffic("other", 10) is None
    with open(dst / "sweep.hpp", "a") as f:
        f.write("\n// changed\n")
    assert bench.stored_traffic("w", 10) is None
