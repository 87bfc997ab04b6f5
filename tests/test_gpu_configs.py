"""GPU parity at the full configuration sizes: the HIP path's calibration,
plan tables and every output byte (by SHA-256 of the NCHW int8 output, plus
sampled values for diagnosis) against the oracle's results stored in
tests/golden/configs.json, which tests/golden/make_golden.py writes from the
oracle alone."""
import hashlib
import json
import os

import numpy as np
import pytest

import paper_2209_12982_amd as W
import workloads

from gpu_util import from_device_nchw, to_device, torch_dev, workspace

pytestmark = pytest.mark.gpu

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "configs.json")))


def _run_layer(x, f, b, spec, rec, layout, variant=W.SPLIT, tap_kernel=W.TAP_AUTO, m=4):
    torch = torch_dev()
    n, cin, h, w = x.shape
    xd = to_device(x, layout)
    calibrate = W.wino_f4_calibrate_input if m == 4 else W.wino_f2_calibrate_input
    make_plan = W.wino_f4_plan if m == 4 else W.wino_f2_plan
    eb, amax = calibrate(xd, n, cin, h, w, layout)
    assert eb == rec["e_b"], "input tap exponents differ from the oracle"
    plan0 = make_plan(f, eb, bias=b, out_shift=0, relu=spec.relu)
    info0 = W.wino_f4_plan_info(plan0)
    assert info0["e_g"] == rec["e_g"] and info0["sh"] == rec["sh"] and info0["e_o"] == rec["e_o"]
    if spec.out_shift is None:
        s, zmax = W.wino_f4_calibrate_output(plan0, xd, n, h, w, layout, workspace(plan0, n, h, w))
        assert zmax == rec["zmax"] and s == rec["out_shift"]
    else:
        s = spec.out_shift
    plan = make_plan(f, eb, bias=b, out_shift=s, relu=spec.relu)
    W.wino_f4_plan_set_tap_kernel(plan, tap_kernel)
    shape = (n, spec.cout, h, w) if layout == W.NCHW else (n, h, w, spec.cout)
    y = torch.full(shape, 77, dtype=torch.int8, device="cuda")
    ws = workspace(plan, n, h, w, variant) if variant == W.SPLIT else None
    W.wino_f4_conv_int8(plan, xd, y, n, h, w, layout, variant, ws)
    torch.cuda.synchronize()
    yn = from_device_nchw(y, layout)
    for idx, v in rec["samples"]:
        assert int(yn[tuple(idx)]) == v, f"sample {idx}: {int(yn[tuple(idx)])} != {v}"
    assert hashlib.sha256(yn.tobytes()).hexdigest() == rec["sha256_nchw"]
    return yn


RUNS = [(W.NHWC, W.SPLIT, W.TAP_AUTO), (W.NCHW, W.SPLIT, W.TAP_AUTO), (W.NHWC, W.FUSED, W.TAP_AUTO),
        (W.NCHW, W.FUSED, W.TAP_AUTO), (W.NHWC, W.SPLIT, W.TAP_RESIDENT_64X32), (W.NCHW, W.SPLIT, W.TAP_ROWS),
        (W.NHWC, W.SPLIT, W.TAP_ROWS), (W.NCHW, W.SPLIT, W.TAP_WAVES), (W.NHWC, W.SPLIT, W.TAP_WAVES),
        (W.NHWC, W.SPLIT, W.TAP_RESIDENT_32X32), (W.NHWC, W.SPLIT, W.TAP_ROWS_STREAMK),
        (W.NCHW, W.SPLIT, W.TAP_ROWS_STREAMK)]


@pytest.mark.parametrize("layout,variant,tap_kernel", RUNS)
@pytest.mark.parametrize("name", ["C4", "C5"])
def test_full_size_layer_bitexact(name, layout, variant, tap_kernel):
    x, layers = workloads.generate(name)
    f, b, spec = layers[0]
    _run_layer(x, f, b, spec, GOLDEN[name]["layers"][0], layout, variant, tap_kernel)


@pytest.mark.parametrize("layout", [W.NCHW, W.NHWC])
@pytest.mark.parametrize("name", ["C1", "C2"])
def test_small_config_bitexact(name, layout):
    """C1 (its literal out_shift 8) and C2 against their full records, SPLIT
    and FUSED."""
    x, layers = workloads.generate(name)
    f, b, spec = layers[0]
    for variant in (W.SPLIT, W.FUSED):
        _run_layer(x, f, b, spec, GOLDEN[name]["layers"][0], layout, variant)


@pytest.mark.parametrize("layout", [W.NCHW, W.NHWC])
@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5"])
def test_f2_first_layer_bitexact(name, layout):
    """F(2x2, 3x3) on every configuration's first layer at full size: the
    GPU's F2 calibration, tables and every output byte against the oracle's
    F2 record."""
    x, layers = workloads.generate(name)
    f, b, spec = layers[0]
    _run_layer(x, f, b, spec, GOLDEN[name]["f2_layers"][0], layout, W.SPLIT, W.TAP_AUTO, m=2)


@pytest.mark.parametrize("layout,variant,tap_kernel", RUNS)
def test_c3_chain_bitexact(layout, variant, tap_kernel):
    """Four chained layers; each layer's input is the GPU's own previous
    output (max-pooled where the stage halves the image), and every layer
    must match the oracle's chain byte for byte."""
    x, layers = workloads.generate("C3")
    cur = x
    for k, (f, b, spec) in enumerate(layers):
        if k > 0:
            cur = workloads.next_layer_input(cur, spec)
        cur = _run_layer(cur, f, b, spec, GOLDEN["C3"]["layers"][k], layout, variant, tap_kernel)
