"""Host-side contract of bench.py: a run on more than one GPU is refused with a
JSON message and exit status 2, before any device is touched."""

import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args, env=None):
    e = dict(os.environ)
    e.update(env or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + args, cwd=ROOT,
                          capture_output=True, text=True, env=e, timeout=120)


def test_more_than_one_gpu_is_refused():
    r = _run(["--gpus", "2", "--steps", "1", "--warmup", "0"])
    assert r.returncode == 2
    out = json.loads(r.stdout.strip().splitlines()[-1])
    assert out["n_gpus"] == 2 and "error" in out


def test_a_second_rank_is_refused():
    r = _run(["--steps", "1"], env={"WORLD_SIZE": "2"})
    assert r.returncode == 2
    assert "error" in json.loads(r.stdout.strip().splitlines()[-1])


def test_cpu_baseline_host_facts():
    """Every CPU baseline records the oracle's threads, the host's CPU count and
    model, and the BLAS library numpy calls."""
    sys.path.insert(0, ROOT)
    import bench
    info = bench.host_info(3)
    assert info["cores"] == 3
    assert info["host_cpus"] == os.cpu_count()
    assert isinstance(info["cpu_model"], str) and info["cpu_model"]
    assert isinstance(info["blas"], str) and info["blas"]
    st = bench.step_stats([3.0, 1.0, 2.0, 10.0])
    assert st["median"] == 2.5 and st["n"] == 4 and st["max"] == 10.0
    assert "36%" in bench.PAPER_CONTEXT["training_compute"]
    assert "14%" in bench.PAPER_CONTEXT["speculative_decoding"]
