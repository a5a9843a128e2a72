"""bench.py's output line on the GPU: one JSON object with the contract's fields, the roofline
entry of the dominant kernel and the oracle's CPU baseline, for the Adam and the LAMB step.
Runs the small 1M-element shard with short timed regions: the Adam step there is the one-launch
small-shard kernel (no counter summary is kept for it, so `traffic` is null), the LAMB step's
dominant kernel its moments pass (its summary is for the 250M shard)."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*extra):
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny", "--steps", "50", "--warmup", "5",
           "--step-samples", "10", "--probe-copy-mib", "64", "--cpu-budget", "0.5", "--cpu-parallel-budget", "0.5",
           *extra]
    print("[gpu-bench-contract]", " ".join(cmd[1:]), flush=True)
    r = subprocess.run(cmd, cwd=ROOT, stdout=subprocess.PIPE, stderr=subprocess.PIPE, timeout=110)
    assert r.returncode == 0, r.stderr.decode(errors="replace")[-2000:]
    lines = [ln for ln in r.stdout.decode().splitlines() if ln.strip()]
    assert len(lines) == 1, lines
    return json.loads(lines[0])


def _check(d, kernel):
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
              "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline", "step_ms_quantiles"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 50 and d["warmup"] == 5
    assert d["unit"] == "params/s" and d["higher_is_better"] is True and d["vs_baseline"] is None
    assert d["data"] == "synthetic" and d["config"]["workload"] == "tiny"
    n = d["config"]["shard_numel"]
    assert abs(d["value"] - n / (d["ms_per_step"] * 1e-3)) <= 1e-6 * d["value"]
    rf = d["roofline"]
    assert rf["bound"] == "hbm" and rf["kernel"] == kernel and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert 0 < rf["achieved"] < rf["peak"] and abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-12
    assert rf["traffic"] is None
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] == 1 and cb["value"] > 0 and cb["unit"] == "params/s"
    q = d["step_ms_quantiles"]
    assert 0 < q["p10"] <= q["p50"] <= q["p90"] and q["steps"] == 10


def test_adam_line():
    d = _run()
    _check(d, "k_small_step")
    assert "adam_probe" not in d  # the one-launch step has no separate update kernel to compare
    cp = d["cpu_baseline_parallel"]
    assert cp["kind"] == "oracle" and cp["cores"] >= 1 and cp["value"] > 0 and cp["unit"] == "params/s"


def test_lamb_line():
    d = _run("--optimizer", "lamb")
    _check(d, "k_lamb_moments")
    assert d["config"]["optimizer"] == "lamb" and d["lamb_apply"]["kernel"] == "k_lamb_apply"


@pytest.mark.parametrize("mode", [("--resident", "eager"), ("--resident", "graph"), ("--split-phase",),
                                  ("--split-phase", "--async-seam")])
def test_other_step_forms_print_their_line(mode):
    # the resident step (eager and graph replays) and the split phase (host or device seam):
    # three kernels per step, the update's roofline entry
    d = _run(*mode)
    _check(d, "k_adam_vec")
    assert "path" in d["config"]
    ap = d["adam_probe"]  # the update's byte-mix probe on the same arrays
    assert ap["kernel"] == "k_probe_adam" and ap["probe_ms"] > 0 and ap["probe_gbps"] > 0
    assert abs(ap["update_frac_of_probe"] - ap["update_gbps"] / ap["probe_gbps"]) < 1e-12
