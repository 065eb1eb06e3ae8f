"""bench.py's command line on the CPU: the refusals that need no GPU."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=300)


def test_more_than_one_gpu_is_refused():
    r = run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU only" in r.stderr


def test_mode_override_only_for_stack_workloads():
    r = run("--workload", "field256", "--mode", "bidir")
    assert r.returncode == 2
    assert "--mode applies to the stack workloads" in r.stderr
