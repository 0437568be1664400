"""Host-side logic of bench.py (no GPU): warm-up and timed-step counts, the
one-GPU guard, and when committed HBM byte counts are reported."""
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


def test_traffic_is_reported_only_for_current_sources(monkeypatch, tmp_path):
    """A counter summary counts only while the hash of the kernel's sources
    and compiler flags still matches the one stored with it."""
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    import json
    for kernel in bench.KERNEL_FILES:
        assert bench.load_traffic(kernel, "w") is None  # nothing taken
        good = {"source_sha256": bench.kernel_source_hash(kernel), "hbm_bytes_per_launch": 123.0}
        with open(bench.traffic_file(kernel, "w"), "w") as fh:
            json.dump(good, fh)
        assert bench.load_traffic(kernel, "w") == 123.0
        with open(bench.traffic_file(kernel, "w"), "w") as fh:
            json.dump(dict(good, source_sha256="0" * 64), fh)
        assert bench.load_traffic(kernel, "w") is None
    hashes = {bench.kernel_source_hash(k) for k in bench.KERNEL_FILES}
    assert len(hashes) == len(bench.KERNEL_FILES)


def test_source_hash_ignores_include_paths(monkeypatch):
    """The hash must be the same on any machine: include paths (which name
    the checkout's location) are left out, other flags are not."""
    from paper_2101_08763_amd import build as B
    h0 = bench.kernel_source_hash("sqnorm_kernel")
    monkeypatch.setattr(B, "FLAGS", [f if not f.startswith("-I") else "-I/elsewhere" for f in B.FLAGS])
    assert bench.kernel_source_hash("sqnorm_kernel") == h0
    monkeypatch.setattr(B, "FLAGS", B.FLAGS + ["-O0"])
    assert bench.kernel_source_hash("sqnorm_kernel") != h0
