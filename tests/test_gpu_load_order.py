"""The library works when its first call in a process comes before any
PyTorch device work (PyTorch's own HIP runtime must be the one the library
binds to; see load_library)."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CHILD = """
import numpy as np
import paper_2209_12982_amd as W
f = np.zeros((4, 4, 3, 3), np.float32)
W.wino_f4_plan(f, [0] * 36)
W.wino_f4_plan_i10(f, [0] * 36)
print("ok")
"""


def test_plan_before_any_torch_device_work():
    env = dict(os.environ, PYTHONPATH=ROOT)
    r = subprocess.run([sys.executable, "-c", CHILD], env=env, capture_output=True, text=True, timeout=110)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
