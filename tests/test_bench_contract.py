"""bench.py's output contract: one JSON line with the metric, the step time,
the roofline entry and the CPU baseline, from a short run of a small workload
(GPU), and a clear refusal of more than one GPU (CPU: it exits before any GPU
work)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args, timeout):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + args, cwd=ROOT,
                          capture_output=True, text=True, timeout=timeout)


def test_more_than_one_gpu_is_refused():
    r = _run(["--gpus", "2"], timeout=120)
    assert r.returncode != 0
    assert "--gpus 2 is not supported" in r.stderr
    assert r.stdout.strip() == ""


@pytest.mark.gpu
def test_json_line(gpu_lib):
    print("[bench] loss4k, 2 steps, 64-row CPU baseline", flush=True)
    r = _run(["--workload", "loss4k", "--steps", "2", "--warmup", "1", "--cpu-rows", "64",
              "--split-steps", "1"], timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1
    rec = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
              "roofline", "cpu_baseline", "mfma_pct", "gemm_flop_per_step"):
        assert k in rec, k
    assert rec["n_gpus"] == 1 and rec["steps"] == 2 and rec["warmup"] == 1
    assert rec["unit"] == "tokens/s" and rec["higher_is_better"] is True
    assert rec["dtype"] == "bf16" and rec["data"] == "synthetic"
    assert rec["config"]["workload"] == "loss4k"
    # value is whole-step tokens/s from the step time
    assert abs(rec["value"] - 4096 / (rec["ms_per_step"] / 1e3)) <= 1e-3 * rec["value"]
    # the fused call executes 6 N D V per step (no mask here)
    assert rec["gemm_flop_per_step"] == pytest.approx(6.0 * 4096 * 4096 * 131072, rel=1e-9)
    rf = rec["roofline"]
    for k in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert k in rf, k
    assert rf["bound"] == "mfma" and rf["unit"] == "TFLOP/s" and rf["peak"] == 2500.0
    assert 0.0 < rf["frac"] < 1.0 and rf["frac"] == pytest.approx(rf["achieved"] / rf["peak"],
                                                                  abs=1e-4)
    cb = rec["cpu_baseline"]
    for k in ("value", "unit", "cores", "kind", "sample"):
        assert k in cb, k
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1
