"""The benchmark's output contract on the GPU: one JSON line with throughput,
the dominant kernel's roofline and the CPU oracle's rate, for every mode.

Short runs (two timed steps, a 16-row oracle sample) of the same code the full
benchmark executes."""

import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
MODES = [[], ["--diagnostics"], ["--junction"], ["--decode"]]


def _run(extra):
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "2", "--warmup", "1",
           "--cpu-rows", "16"] + extra
    print("[bench-contract]", " ".join(extra) or "fwd+bwd", flush=True)
    r = subprocess.run(cmd, cwd=ROOT, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [x for x in r.stdout.splitlines() if x.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    return json.loads(lines[0])


@pytest.mark.parametrize("extra", MODES, ids=["main", "diagnostics", "junction", "decode"])
def test_bench_line_contract(extra):
    out = _run(extra)
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config"):
        assert k in out, k
    assert out["n_gpus"] == 1 and out["steps"] == 2 and out["warmup"] == 1
    assert out["value"] > 0 and out["ms_per_step"] > 0 and out["higher_is_better"] is True
    assert "workload" in out["config"]
    roof = out["roofline"]
    assert roof["bound"] in ("hbm", "mfma", "alu")
    assert roof["unit"] in ("GB/s", "TFLOP/s")
    assert 0 < roof["achieved"] and 0 < roof["peak"]
    assert abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-9
    assert roof["traffic"] is None or roof["traffic"] > 0
    cpu = out["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["value"] > 0 and cpu["cores"] >= 1
    assert cpu["unit"] == out["unit"] and cpu["sample"]
    for k in ("host_cpus", "cpu_model", "blas"):
        assert k in cpu, k
    assert "paper_context" in out
    if "ms_per_step_stats" in out:
        assert out["ms_per_step"] == out["ms_per_step_stats"]["median"]
