"""Host-side pieces of bench.py: the work and ceiling formulas behind its roofline fields, and the
one-GPU contract.  No GPU is touched."""
import math
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("block,want", [(1, 1), (5, 1), (6, 2), (16, 2), (21, 2), (22, 3), (256, 17), (257, 17),
                                        (261, 17), (262, 18)])
def test_compressions_per_key(block, want):
    # message of one key: 16 B previous key + 16 B digest + 4B bytes of tokens, plus at least 9 bytes
    # of padding, in 64-byte blocks
    assert bench.compressions_per_key(block) == want == math.ceil((32 + 4 * block + 9) / 64)


def test_ceilings_scale_with_chains_and_stop_at_one():
    # one chain: 1384 lane-ops per 64 rounds; at most one round per 16 cycles (dependence) or per
    # 40 cycles (the 10-instruction round), against 256 CUs x 64 lanes per clock
    per_lane_clock = 256 * 64
    assert bench.chain_ceiling_frac(1) == pytest.approx(1384 / (64 * 16) / per_lane_clock)
    assert bench.issue_ceiling_frac(1) == pytest.approx(1384 / (64 * 40) / per_lane_clock)
    assert bench.chain_ceiling_frac(1024) == pytest.approx(0.08447, abs=1e-5)
    assert bench.issue_ceiling_frac(1024) == pytest.approx(0.03379, abs=1e-5)
    assert bench.chain_ceiling_frac(10 ** 6) == 1.0 and bench.issue_ceiling_frac(10 ** 6) == 1.0
    assert bench.issue_ceiling_frac(4096) < bench.chain_ceiling_frac(4096)


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_default_workload_is_the_largest_configuration():
    # 16384 requests x 4096 tokens against the 2^26-slot index is the largest specified shape
    import argparse
    old = sys.argv
    try:
        sys.argv = ["bench.py"]
        args = bench.parse()
    finally:
        sys.argv = old
    assert args.workload == "c4" and args.gpus == 1


def test_cpu_threads_stay_within_the_one_gpu_share():
    class A:
        cpu_threads = 0
    t, host = bench.cpu_threads(A())
    assert 1 <= t <= bench.CPU_SHARE and t <= host == len(os.sched_getaffinity(0))
    A.cpu_threads = 3
    assert bench.cpu_threads(A())[0] == 3
