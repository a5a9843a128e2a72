"""bench.py's contract pieces that need no GPU: it refuses more than one GPU with a
message, and it reads the committed counter summaries (Adam update, LAMB moments pass) only
for the kernels and launch policy they were taken on."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import pytest  # noqa: E402

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], stdout=subprocess.PIPE,
                       stderr=subprocess.PIPE, timeout=120)
    assert r.returncode == 2
    assert b"one GPU" in r.stderr and r.stdout == b""


@pytest.mark.parametrize("workload,n", [("gpt2_1p5b", 93_750_000), ("dp_13b", 203_125_000),
                                        ("mp16_dp25_100b", 250_000_000), ("ragged_1t", 61_034_389)])
def test_traffic_summary_matches_the_kernel_sources_or_is_ignored(tmp_path, monkeypatch, workload, n):
    t = bench.measured_traffic(workload, n)
    if t is not None:  # present and current: it must be close to the 28 B/element algorithmic bytes
        assert abs(t / (28 * n) - 1) < 0.01
    assert bench.measured_traffic(workload, 12345) is None  # another shard size
    assert bench.measured_traffic("tiny", 1_048_576) is None  # no summary for that workload
    stale = tmp_path / "t_%s.txt"
    (tmp_path / ("t_%s.txt" % workload)).write_text(
        "kernel_source_sha256_16: 0000\nshard_numel: %d\nupdate_bytes_per_launch: 7e9\n" % n)
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(stale))
    assert bench.measured_traffic(workload, n) is None  # taken on other kernels
    (tmp_path / ("g_%s.txt" % workload)).write_text("kernel_source_sha256_16: %s\nshard_numel: %d\n"
                                                   "update_bytes_per_launch: 7e9\n" % (bench.kernel_source_hash(), n))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "g_%s.txt"))
    assert bench.measured_traffic(workload, n) == 7e9


def test_committed_traffic_summaries_match_the_current_kernels():
    # the counter summaries under profiles/ were taken on the kernel sources as they stand, so the
    # bench line carries measured traffic for every large workload (a kernel change needs new counters)
    for workload, n in (("gpt2_1p5b", 93_750_000), ("dp_13b", 203_125_000), ("mp16_dp25_100b", 250_000_000),
                        ("ragged_1t", 61_034_389)):
        assert bench.measured_traffic(workload, n) is not None, workload
    assert bench.measured_lamb_traffic(250_000_000) is not None


def test_lamb_traffic_summary_matches_the_kernel_sources_or_is_ignored(tmp_path, monkeypatch):
    t = bench.measured_lamb_traffic(250_000_000)
    if t is not None:  # present and current: within 1 % of the moments pass's 22 B/element
        assert abs(t / (22 * 250_000_000) - 1) < 0.01
    assert bench.measured_lamb_traffic(12345) is None
    stale = tmp_path / "t.txt"
    stale.write_text("kernel_source_sha256_16: %s\nshard_numel: 250000000\nmoments_bytes_per_launch: 5.5e9\n"
                     % bench.kernel_source_hash())  # the Adam hash is not the LAMB kernels' hash
    monkeypatch.setattr(bench, "LAMB_TRAFFIC_FILE", str(stale))
    assert bench.measured_lamb_traffic(250_000_000) is None
    good = tmp_path / "g.txt"
    good.write_text("kernel_source_sha256_16: %s\nshard_numel: 250000000\nmoments_bytes_per_launch: 5.5e9\n"
                    % bench.lamb_kernel_source_hash())
    monkeypatch.setattr(bench, "LAMB_TRAFFIC_FILE", str(good))
    assert bench.measured_lamb_traffic(250_000_000) == 5.5e9


def test_kernel_hashes_ignore_comments_but_not_code():
    src = "int a = 1; // one\n/* block */ int b = 2;\n\n"
    assert bench._code_only(src) == bench._code_only("int a = 1;\nint b = 2;")
    assert bench._code_only(src) != bench._code_only("int a = 1;\nint b = 3;")
