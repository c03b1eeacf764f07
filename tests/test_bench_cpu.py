"""Host-side logic of bench.py (no GPU): the launch count of a sweep solve
that the roofline divides by, the one-GPU contract, and the traffic gate."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _schedule(p, s):
    """The step schedule written out: blocks of 64 columns, a step making
    SWEEP_STEP_BLOCKS blocks final (the last step the rest)."""
    nblk = -(-p // 64)
    steps, t = [], 0
    while t < nblk:
        nb = min(bench.SWEEP_STEP_BLOCKS, nblk - t)
        steps.append((t, nb))
        t += nb
    return nblk, steps


@pytest.mark.parametrize("p,s", [(261755, 32), (1042161, 64), (261755, 16), (1000, 32), (64, 8),
                                 (65, 8), (131200, 32)])
def test_sweep_launches_cover_every_block_once(p, s):
    nblk, steps = _schedule(p, s)
    assert bench.sweep_launches(p, s) == len(steps)
    made = [b for t, nb in steps for b in range(t, t + nb)]
    assert made == list(range(nblk))


def test_default_workload_launch_count():
    # 4090 blocks of 64 columns, twelve per launch
    assert bench.sweep_launches(261755, 32) == 341


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_reported_only_for_its_workload():
    base = bench.sweep_roofline(261755, 32, 100.0, 1, 1.0, measured=True)
    other = bench.sweep_roofline(261755, 32, 100.0, 1, 1.0, measured=False)
    assert other["traffic"] is None
    if bench.kernel_sources_sha(bench.SWEEP_SOURCES) == bench.SWEEP_TRAFFIC_SHA:
        assert base["traffic"] == bench.SWEEP_TRAFFIC_BYTES_PER_LAUNCH
    else:
        assert base["traffic"] is None
