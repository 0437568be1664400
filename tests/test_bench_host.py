"""Host-side logic of bench.py (no GPU): warm-up and timed-step counts, and
the one-GPU guard."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_explicit_warmup_runs_exactly():
    calls, syncs = [], []
    n, per = bench.warm_up(lambda: calls.append(1), 7, lambda: syncs.append(1))
    assert n == 7 and len(calls) == 7 and per >= 0


def test_zero_warmup_is_allowed():
    calls = []
    n, _ = bench.warm_up(lambda: calls.append(1), 0, lambda: None)
    assert n == 0 and calls == []


def test_default_warmup_is_time_based(monkeypatch):
    calls = []
    n, per = bench.warm_up(lambda: calls.append(1), None, lambda: None, seconds=0.05)
    assert n == len(calls) and n >= bench.MIN_WARMUP
    assert n * per >= 0.05


def test_timed_steps():
    assert bench.timed_steps(3, 1.0) == 3                     # explicit: exactly
    assert bench.timed_steps(None, 1.0) == bench.MIN_STEPS    # slow steps: the minimum
    assert bench.timed_steps(None, 1e-4) >= bench.TIMED_SECONDS / 1e-4
    assert bench.timed_steps(None, 1.0, min_steps=3) == 3


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
