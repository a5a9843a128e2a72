"""bench.py's contract pieces that need no GPU: it refuses more than one GPU with a
message, and it reads the committed counter summary only for the current kernels."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], stdout=subprocess.PIPE,
                       stderr=subprocess.PIPE, timeout=120)
    assert r.returncode == 2
    assert b"one GPU" in r.stderr and r.stdout == b""


def test_traffic_summary_matches_the_kernel_sources_or_is_ignored(tmp_path, monkeypatch):
    t = bench.measured_traffic(250_000_000)
    if t is not None:  # present and current: it must be close to the 28 B/element algorithmic bytes
        assert abs(t / (28 * 250_000_000) - 1) < 0.01
    assert bench.measured_traffic(12345) is None  # another shard size
    stale = tmp_path / "t.txt"
    stale.write_text("kernel_source_sha256_16: 0000\nshard_numel: 250000000\nupdate_bytes_per_launch: 7e9\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(stale))
    assert bench.measured_traffic(250_000_000) is None  # taken on other kernels
    good = tmp_path / "g.txt"
    good.write_text("kernel_source_sha256_16: %s\nshard_numel: 250000000\nupdate_bytes_per_launch: 7e9\n"
                    % bench.kernel_source_hash())
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(good))
    assert bench.measured_traffic(250_000_000) == 7e9
