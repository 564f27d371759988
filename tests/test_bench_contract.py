"""Host-side parts of bench.py: the one-GPU guard, the traffic record lookup
and the bounded timing loop of the CPU baseline (no GPU needed)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


@pytest.mark.parametrize("kernel", sorted(bench.KERNEL_SOURCES))
def test_traffic_record_is_used_only_for_unchanged_sources(kernel, monkeypatch):
    with open(bench.TRAFFIC_FILE) as f:
        rec = {p[1]: (int(p[2]), p[3]) for p in (l.split() for l in f)
               if len(p) == 4 and p[0] == "traffic"}
    assert kernel in rec
    nbytes, digest = rec[kernel]
    monkeypatch.setattr(bench, "source_digest", lambda k: digest)
    assert bench.measured_traffic(kernel) == nbytes
    monkeypatch.setattr(bench, "source_digest", lambda k: "0" * 16)
    assert bench.measured_traffic(kernel) is None
    assert bench.measured_traffic("no_such_kernel") is None


def test_timed_calls_stops_at_the_budget_or_the_call_cap():
    n = []
    calls, el = bench.timed_calls(lambda: n.append(1), 0.05)
    assert calls == len(n) == 1000 and el < 5.0     # cheap calls: the cap ends the loop
    import time
    calls, el = bench.timed_calls(lambda: time.sleep(0.02), 0.05)
    assert 1 <= calls <= 4 and el >= 0.05
    one = bench.single_thread_rate(lambda: None, 0.01)
    assert one is None or one[0] >= 1
