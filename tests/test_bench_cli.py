"""bench.py's command line (CPU): the workload each mode runs by default, and
the refusal of more than one GPU before anything touches a device."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


@pytest.mark.parametrize("argv, workload", [
    ([], "70b-gqa-b128-L8192"),                           # the largest configuration
    (["--model", "llama2-7b"], "7b-b64-L4096"),           # whole layers need 32 heads of 128
    (["--no-pd"], "b32-L2048"),                           # the ring widens by each step's longest prompt
    (["--no-pd", "--config", "7b-b64-L4096"], "7b-b64-L4096"),
])
def test_default_workloads(monkeypatch, argv, workload):
    monkeypatch.setattr(sys, "argv", ["bench.py"] + argv)
    assert bench.parse().config == workload


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""
