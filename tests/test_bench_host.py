"""bench.py's contract on a host without a GPU: it measures one GPU only, says
so for any other count, fails plainly when no GPU is visible, and reports
counter-measured HBM traffic only for the kernel source and workload the
committed counters were taken on."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _run(*args):
    env = dict(os.environ, HIP_VISIBLE_DEVICES="", CUDA_VISIBLE_DEVICES="")
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True,
                          text=True, timeout=300, env=env, cwd=ROOT)


@pytest.mark.parametrize("n", ["2", "8"])
def test_more_than_one_gpu_is_refused_with_a_message(n):
    res = _run("--gpus", n)
    assert res.returncode == 2
    assert "one GPU" in res.stderr and res.stdout == ""


def test_no_visible_gpu_fails_without_a_result_line():
    res = _run("--steps", "1", "--warmup", "0", "--no-cpu-baseline")
    assert res.returncode != 0
    assert not any(line.startswith("{") for line in res.stdout.splitlines())


def _counters(tmp_path, sha, workload="resnet50", traffic="1278312108"):
    p = tmp_path / "counters.txt"
    p.write_text("# header line: ignored\n"
                 f"workload: {workload}\n"
                 f"kernel_source_sha256_16: {sha}\n"
                 f"traffic_bytes_per_launch: {traffic}\n")
    return str(p)


def test_traffic_is_reported_only_for_the_profiled_source_and_workload(tmp_path, monkeypatch):
    sha = bench.kernel_source_sha()
    monkeypatch.setattr(bench, "COUNTERS_FILE", _counters(tmp_path, sha))
    assert bench.counter_traffic("resnet50") == 1278312108.0
    assert bench.counter_traffic("segnet") is None                     # another workload
    monkeypatch.setattr(bench, "COUNTERS_FILE", _counters(tmp_path, "0" * 16))
    assert bench.counter_traffic("resnet50") is None                   # taken on other kernels
    monkeypatch.setattr(bench, "COUNTERS_FILE", str(tmp_path / "missing.txt"))
    assert bench.counter_traffic("resnet50") is None


def test_kernel_source_hash_follows_the_kernel_sources(tmp_path, monkeypatch):
    a = tmp_path / "a.hip"
    a.write_text("kernel text\n")
    monkeypatch.setattr(bench, "KERNEL_SOURCES", [str(a)])
    h0 = bench.kernel_source_sha()
    a.write_text("kernel text, one comment changed\n")
    assert bench.kernel_source_sha() != h0 and len(h0) == 16


def test_committed_counters_match_the_algorithmic_bytes():
    """When the committed counter summary was taken on the current sources, its
    traffic is the resnet50-shaped step's algorithmic bytes within 1% (no
    stream read twice); otherwise the bench reports traffic as null."""
    t = bench.counter_traffic("resnet50")
    if t is None:
        pytest.skip("counters were taken on another kernel source: the bench reports traffic null")
    algorithmic = 25_557_032 * 50
    assert algorithmic <= t <= 1.01 * algorithmic
