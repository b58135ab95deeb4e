"""Host-side contract of bench.py: a run on more than one GPU is refused with a
JSON message and exit status 2, before any device is touched; the roofline's
traffic figure is read from the committed summaries only while they match the
kernel sources."""

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


def test_profiled_traffic_follows_the_kernel_sources(tmp_path, monkeypatch):
    """roofline.traffic comes from a committed summary only while its recorded hash
    of the kernel sources matches; each kind of run reads its own summary."""
    sys.path.insert(0, ROOT)
    import bench
    (tmp_path / "profiles").mkdir()
    block = {"sources_sha256": "abc", "per_launch": {"gemm_grads": {"fetch_bytes": 3.0, "write_bytes": 4.0}}}
    for kind in ("kernels", "recompute"):
        (tmp_path / "profiles" / f"w_{kind}.md").write_text(
            "# summary\n\n```json\n" + json.dumps(block) + "\n```\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "sources_sha256", lambda: "abc")
    assert bench.profiled_traffic("w", "gemm_grads") == 7.0
    assert bench.profiled_traffic("w", "gemm_grads", "recompute") == 7.0
    assert bench.profiled_traffic("w", "fused_fwd") is None          # kernel not in the summary
    assert bench.profiled_traffic("w", "gemm_grads", True) is None   # no diagnostics summary
    monkeypatch.setattr(bench, "sources_sha256", lambda: "changed")
    assert bench.profiled_traffic("w", "gemm_grads") is None


def test_committed_summaries_match_the_kernel_sources():
    """Every committed summary records the hash of the kernel sources it was taken
    on; all of them are current."""
    sys.path.insert(0, ROOT)
    import re
    import bench
    names = sorted(os.listdir(os.path.join(ROOT, "profiles")))
    assert len(names) >= 7
    for n in names:
        m = re.search(r"```json\n(.*?)\n```", open(os.path.join(ROOT, "profiles", n)).read(), re.S)
        assert m, n
        assert json.loads(m.group(1))["sources_sha256"] == bench.sources_sha256(), n
