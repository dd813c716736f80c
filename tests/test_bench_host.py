"""Host-side logic of bench.py (no GPU): the multi-GPU refusal, the clock
settling rule and the HBM-traffic summary lookup."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    assert "multi-GPU" in r.stderr
    assert r.stdout.strip() == ""


@pytest.mark.parametrize("means, calls, expect", [
    ([0.688, 0.484], 20, False),                        # too few calls
    ([0.405, 0.405], 140, False),                       # steady, still below the minimum
    ([0.420, 0.405], 150, False),                       # 3.6 % apart
    ([0.4080, 0.4050], 150, True),                      # 0.7 % apart
    ([0.4050, 0.4090], 500, True),                      # 1.0 %: at the tolerance
    ([0.405], 150, False),                              # one chunk: nothing to compare
])
def test_settling_rule(means, calls, expect):
    assert bench.settled(means, calls) is expect


def test_traffic_summary_is_read_only_for_its_sources():
    t = bench.measured_traffic()
    text = open(os.path.join(ROOT, bench.TRAFFIC_SUMMARY)).read()
    if "gemm source hash: " + bench.gemm_source_hash() in text:
        assert isinstance(t, int) and t > 0
    else:
        assert t is None
