"""bench.py's command-line contract on the CPU: it measures one GPU and says
so for --gpus above 1, and --chain only times the C3 stack.  Both refusals
happen before anything touches a GPU."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=300)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stdout + r.stderr
    assert r.stdout.strip() == "" or not r.stdout.lstrip().startswith("{")


def test_chain_needs_c3():
    r = _run("--chain", "--config", "C5")
    assert r.returncode == 2
    assert "C3" in r.stderr
