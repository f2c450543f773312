"""Host-side parts of bench.py that need no GPU: the one-GPU guard and the
rule that the convolution's HBM traffic figure is reported only for the
kernel source it was measured on."""
import hashlib
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


@pytest.mark.parametrize("argv, env", [(["--gpus", "2"], {}), (["--gpus", "1"], {"WORLD_SIZE": "4"})])
def test_more_than_one_gpu_exits_with_a_message(argv, env):
    run = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv],
                         env={**os.environ, **env}, capture_output=True, text=True, timeout=120)
    assert run.returncode == 2
    assert "exactly one GPU" in run.stderr
    assert run.stdout == ""  # no JSON line for a run that did not happen


def test_traffic_only_for_the_profiled_source(tmp_path, monkeypatch):
    src = tmp_path / "kernel.hip"
    src.write_text("// one version\n")
    sha = hashlib.sha256(src.read_bytes()).hexdigest()[:16]
    monkeypatch.setattr(bench, "CONV_SOURCES", [str(src)])
    monkeypatch.setattr(bench, "CONV_TRAFFIC", {"w": {"bytes": 123, "kernel_sha256": sha}})
    assert bench.conv_traffic("w") == 123
    assert bench.conv_traffic("other workload") is None
    src.write_text("// another version\n")
    assert bench.conv_traffic("w") is None


def test_recorded_traffic_is_at_least_the_algorithmic_bytes():
    # x + out of the imagenet_stage layer in bf16 (64 x 56 x 56 pixels, 256
    # reals each), the four shared kernels aside
    algorithmic = 2 * 64 * 56 * 56 * 256 * 2
    entry = bench.CONV_TRAFFIC["imagenet_stage"]
    assert entry["bytes"] >= algorithmic
    assert len(entry["kernel_sha256"]) == 16
