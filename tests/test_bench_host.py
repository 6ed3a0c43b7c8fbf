"""Host-side checks of bench.py's reporting: the counter summaries it reads
for `roofline.traffic` and the one-GPU guard. No GPU is touched."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402

SHAPES = {"memscale": (10**9, 32), "large": (25_000_000, 32)}


@pytest.mark.parametrize("name", sorted(SHAPES))
def test_counter_summary_is_well_formed(name):
    text = open(bench.PMC_SUMMARIES[name]).read()
    P, K = SHAPES[name]
    assert f"shape: P={P} K={K}" in text
    assert "source_hash:" in text and "hbm_bytes_per_launch:" in text
    # the command that made it runs committed files only
    assert "rocprofv3 --pmc FETCH_SIZE" in text and "rocprofv3 --pmc WRITE_SIZE" in text
    assert "_work" not in text


@pytest.mark.parametrize("name", sorted(SHAPES))
def test_traffic_only_for_its_own_shape(name):
    P, K = SHAPES[name]
    assert bench.measured_traffic(name, P, K + 1) is None
    assert bench.measured_traffic(name, P + 1, K) is None
    assert bench.measured_traffic("mlp", P, K) is None
    assert bench.measured_traffic(name, P, K, math="ieee") is None
    got = bench.measured_traffic(name, P, K)
    text = open(bench.PMC_SUMMARIES[name]).read()
    if f"source_hash: {bench.dense_source_hash()}" in text:
        # counters within a few percent of the algorithmic bytes stated beside them
        assert got is not None and got > 0
    else:
        assert got is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_fetch_copy_rule_follows_the_header():
    # by segments only when the copy does not fit the 256 MB Infinity Cache and
    # most segments hold an entry (a transmitted fraction of a few percent)
    P = 1_000_000_000
    assert bench.fetch_copy_by_segments(P, P // 10)
    assert not bench.fetch_copy_by_segments(P, P // 100)
    assert not bench.fetch_copy_by_segments(25_000_000, 2_500_000)


def test_grouped_timing_reports_the_median_group():
    """Back-to-back figures: one untimed call, then five groups of n calls
    between two events each; the per-call median of the groups and their
    range.  A clock that advances 1 per event and 0.5 per call, with one slow
    group, stands in for the GPU."""
    import types

    class Event:
        now = 0.0

        def __init__(self, enable_timing=True):
            self.at = None

        def record(self):
            Event.now += 1.0
            self.at = Event.now

        def elapsed_time(self, end):
            return end.at - self.at

    calls = [0]

    def fn():
        calls[0] += 1
        Event.now += 0.5 if calls[0] != 30 else 100.5     # call 30 falls in the third group

    fake = types.SimpleNamespace(cuda=types.SimpleNamespace(Event=Event, synchronize=lambda: None))
    ms, (lo, hi) = bench.grouped_b2b(fake, fn, 10)
    assert calls[0] == 1 + 5 * 10
    assert ms == pytest.approx(0.6) and lo == pytest.approx(0.6) and hi == pytest.approx(10.6)
