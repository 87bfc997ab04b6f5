"""GPU test of wino_f4_conv_int8_noalloc, the SPLIT convolution that
allocates nothing (its input-transform workspace is the library's own
per-device array): through the C ABI it must give, byte for byte, what
wino_f4_conv_int8 gives with a caller workspace -- on two calls in a row, the
second with a smaller input, so the second call runs on an array the first one
filled -- and refuse a layer whose workspace exceeds the array before any
device work."""
import hashlib
import json
import os

import numpy as np
import pytest

import paper_2209_12982_amd as W
import workloads
from oracle import tapwise

from gpu_util import empty_out, from_device_nchw, to_device, torch_dev, workspace

pytestmark = pytest.mark.gpu

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "configs.json")))


def _both(plan, x, layout):
    torch = torch_dev()
    n, cin, h, w = x.shape
    xd = to_device(x, layout)
    y_ws = empty_out(n, plan.cout, h, w, layout)
    y_na = empty_out(n, plan.cout, h, w, layout)
    W.wino_f4_conv_int8(plan, xd, y_ws, n, h, w, layout, W.SPLIT, workspace(plan, n, h, w))
    W.wino_f4_conv_int8_noalloc(plan, xd, y_na, n, h, w, layout)
    torch.cuda.synchronize()
    return from_device_nchw(y_ws, layout), from_device_nchw(y_na, layout)


@pytest.mark.parametrize("layout", [W.NHWC, W.NCHW])
def test_noalloc_equals_workspace_entry_large_then_small(layout):
    # first call: the full C5 layer (a 59 MB workspace, near the array's
    # 64 MiB); second call: a small ragged layer on the array the first left
    x, layers = workloads.generate("C5")
    f, b, spec = layers[0]
    rec = GOLDEN["C5"]["layers"][0]
    plan = W.wino_f4_plan(f, rec["e_b"], bias=b, out_shift=rec["out_shift"], relu=spec.relu)
    n, _, h, w = x.shape
    assert W.wino_f4_workspace_bytes(plan, n, h, w, W.SPLIT) <= W.NOALLOC_SCRATCH_BYTES
    ref, got = _both(plan, x, layout)
    assert (got == ref).all(), f"{(got != ref).sum()} bytes differ from the workspace entry point"
    assert hashlib.sha256(got.tobytes()).hexdigest() == rec["sha256_nchw"]

    x2, f2, b2 = workloads.random_case(11, 2, 70, 40, 13, 19, signed=True)
    eb2 = tapwise.calibrate_input_exps(x2)
    plan2 = W.wino_f4_plan(f2, eb2, bias=b2, out_shift=9, relu=True)
    ref2, got2 = _both(plan2, x2, layout)
    assert (got2 == ref2).all(), f"{(got2 != ref2).sum()} bytes differ from the workspace entry point"
    assert (got2 == tapwise.conv_int8(x2, tapwise.make_plan(f2, eb2, bias=b2, out_shift=9, relu=True))).all()


def test_noalloc_refuses_a_workspace_beyond_the_array():
    torch = torch_dev()
    f = np.random.default_rng(5).normal(0, 0.05, (256, 256, 3, 3)).astype(np.float32)
    plan = W.wino_f4_plan(f, [4] * 36, bias=None, out_shift=11)
    n, h, w = 8, 160, 160       # 36 x 12800 tiles x 256 channels = 118 MB of workspace
    assert W.wino_f4_workspace_bytes(plan, n, h, w, W.SPLIT) > W.NOALLOC_SCRATCH_BYTES
    x = torch.zeros((n, h, w, 256), dtype=torch.int8, device="cuda")
    y = torch.full((n, h, w, 256), 77, dtype=torch.int8, device="cuda")
    with pytest.raises(W.WinoError) as e:
        W.wino_f4_conv_int8_noalloc(plan, x, y, n, h, w, W.NHWC)
    assert e.value.status == -5   # WINO_EWORKSPACE
    torch.cuda.synchronize()
    assert int((y != 77).sum()) == 0, "nothing may be written when the call is refused"
