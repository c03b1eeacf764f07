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
    # 4090 blocks of 64 columns, sixteen per launch
    assert bench.sweep_launches(261755, 32) == 256


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


@pytest.mark.parametrize("p,s", [(5, 3), (17, 8), (70, 40), (200, 32)])
def test_roofline_flops_are_the_enumerated_cells(p, s):
    """The roofline's flop count written out cell by cell: every (k, j) pair
    (k < j) costs FLOPS_PAIR, every layer-2 column FLOPS_LAYER2_COL, and every
    (k, j, layer) cell of layers 3..min(s, p) with i - 2 <= k < j
    (j >= i - 1) FLOPS_CELL."""
    pairs = sum(1 for j in range(p) for k in range(j))
    cells = sum(1 for i in range(3, min(s, p) + 1)
                for j in range(i - 1, p) for k in range(i - 2, j))
    want = bench.FLOPS_PAIR * pairs + bench.FLOPS_CELL * cells + bench.FLOPS_LAYER2_COL * (p - 1)
    r = bench.sweep_roofline(p, s, 1.0, 1, 0, measured=False)
    assert r["flops_per_solve"] == want
    assert r["frac"] == pytest.approx(want / 1e-3 / 1e12 / bench.FP64_VECTOR_PEAK_TFLOPS)


def test_issue_bound_ceiling_covers_the_profiled_rate():
    """The flop fraction at full VALU issue for the profiled instruction
    stream lies above the fraction at the profiled time, by the profiled
    VALU busy share."""
    p, s = 261755, 32
    r = bench.sweep_roofline(p, s, 128.35 * 10, 10, 0, measured=True)
    if r["counters"] is None:
        pytest.skip("profile constants are for other kernel sources")
    ceil = r["counters"]["frac_at_full_valu_issue"]
    assert r["frac"] < ceil < 1.0
    assert r["frac"] / ceil == pytest.approx(bench.SWEEP_COUNTER_VALU_BUSY, abs=0.01)
