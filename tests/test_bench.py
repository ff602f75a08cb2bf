"""bench.py end to end on the GPU: one JSON line with the measurement fields.

A short run on the small c2 workload (a few timed steps, a bounded oracle
sample), checked for the fields and their consistency: the value is the
query-heads of a step over its time, the roofline's achieved rate is its
flops over the kernel's time, and the CPU baseline is the oracle's.
"""
import json
import os
import subprocess
import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]


def run_bench(*args):
    env = dict(os.environ)
    r = subprocess.run([sys.executable, str(ROOT / "bench.py"), *args], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=110)
    return r


@pytest.mark.gpu
def test_bench_line_fields():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print("\n[case] bench.py --workload c2 --steps 5 --warmup 3 --warmup-ms 50", flush=True)
    r = run_bench("--workload", "c2", "--steps", "5", "--warmup", "3", "--warmup-ms", "50",
                  "--cpu-seconds", "0.2", "--cpu-max-passes", "1")
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout
    j = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
              "roofline", "cpu_baseline"):
        assert k in j, k
    assert j["n_gpus"] == 1 and j["steps"] == 5 and j["warmup"] == 3
    # the clock pre-heat before the warm-up steps is reported on its own
    assert j["preheat"]["ms"] == 50 and j["preheat"]["steps"] >= 10
    assert j["dtype"] == "bf16" and j["data"] == "synthetic"
    c = j["config"]
    qh = c["B"] * c["H"] * c["N"]
    assert j["value"] == pytest.approx(qh / (j["ms_per_step"] * 1e-3), rel=1e-9)
    rf = j["roofline"]
    assert rf["bound"] == "mfma" and rf["unit"] == "TFLOP/s" and rf["peak"] == 2500.0
    flops = 4.0 * c["d"] * (c["M0"] + c["P"] * c["Ch"]) * qh
    t = j["kernels_ms"]["attention_fwd"]
    assert rf["achieved"] == pytest.approx(flops / (t * 1e-3) / 1e12, rel=1e-9)
    assert rf["frac"] == pytest.approx(rf["achieved"] / rf["peak"], rel=1e-9)
    # the entry points' event times add up to at most the wall time per step
    assert sum(j["kernels_ms"].values()) <= j["ms_per_step"] * 1.05
    cb = j["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1


def test_bench_refuses_more_gpus():
    """Runs on the CPU: the check comes before any GPU use."""
    r = run_bench("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr
