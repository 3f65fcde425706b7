"""Host-side behaviour of bench.py that needs no GPU: the one-GPU contract
and the default warm-up per mode."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


@pytest.mark.parametrize("argv,warmup", [([], 200), (["--workload", "flux_mlp"], 100),
                                         (["--workload", "flux_single"], 20), (["--workload", "flux_stack"], 3),
                                         (["--ablation"], 20), (["--numerics"], 20), (["--dit"], 3),
                                         (["--warmup", "7"], 7), (["--dit", "--warmup", "1"], 1)])
def test_default_warmup(monkeypatch, argv, warmup):
    monkeypatch.setattr(sys, "argv", ["bench.py"] + argv)
    args = bench.parse()
    assert bench.resolve_warmup(args) == warmup
