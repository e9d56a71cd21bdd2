"""Host-side checks of bench.py (no GPU): the multi-GPU request is refused with a message,
and the HBM traffic figure is taken from the committed profile only while the kernel source
it was measured on is unchanged; the clock-settle run lasts as long as asked."""
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "single GPU" in r.stderr


def test_traffic_figure_tracks_the_kernel_source():
    for w in ("llada", "dream", "batched"):
        path = bench.TRAFFIC_SUMMARY.format(workload=w)
        if not os.path.exists(path):
            assert bench.measured_traffic(w) is None
            continue
        text = open(path).read()
        m = re.search(r"^traffic_bytes_per_launch:\s*(\d+)\s+workload:\s*(\w+)\s+source:\s*(\w+)",
                      text, flags=re.M)
        assert m, "the profile must carry its machine-readable line"
        assert m.group(2) == w
        got = bench.measured_traffic(w)
        if m.group(3) == bench.kernel_source_hash():
            assert got == int(m.group(1))
        else:
            assert got is None
    assert bench.measured_traffic("no-such-workload") is None


def test_clock_settle_runs_for_the_requested_time():
    """The settle run before the warm-up calls the step for at least the requested wall time,
    waiting for the queued work every 16 calls, and not at all for 0 ms."""
    import time

    calls, syncs = [], []
    assert bench.settle_clocks(lambda: calls.append(1), 0.0, sync=lambda: syncs.append(1)) == 0
    assert not calls and not syncs
    t0 = time.perf_counter()
    n = bench.settle_clocks(lambda: calls.append(1), 20.0, sync=lambda: syncs.append(1))
    assert time.perf_counter() - t0 >= 0.020
    assert n == len(calls) and n >= 16 and n % 16 == 0
    assert len(syncs) == n // 16
