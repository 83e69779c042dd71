"""Host logic of bench.py: its argument parser and launch plan accept the
driver's command line (no GPU needed)."""
from __future__ import annotations

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
