"""GPU parity of the F(2x2, 3x3) path (plans from wino_f2_plan) through the C
ABI against the oracle's F2 pipeline, bit for bit, for both variants (SPLIT:
input transform to a workspace, then the tap GEMM; FUSED: one kernel)."""
import numpy as np
import pytest

import paper_2209_12982_amd as W
import workloads
from oracle import tapwise

from gpu_util import from_device_nchw, run_conv, to_device, torch_dev, workspace

pytestmark = pytest.mark.gpu

LAYOUTS = [W.NCHW, W.NHWC]

SHAPES = [
    # n, cin, cout, h, w
    (1, 1, 1, 1, 1),
    (1, 3, 5, 7, 9),
    (2, 16, 16, 8, 8),
    (1, 64, 64, 17, 13),
    (2, 70, 80, 12, 30),
    (1, 130, 33, 5, 66),
    (3, 8, 100, 2, 3),
    (1, 256, 64, 14, 14),
]


def _pair(f, eb, b, out_shift, relu, e_g=None):
    gp = W.wino_f2_plan(f, eb, w_exp=e_g, bias=b, out_shift=out_shift, relu=relu)
    op = tapwise.make_plan(f, eb, e_g=e_g, bias=b, out_shift=out_shift, relu=relu, m=2)
    return gp, op


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", SHAPES)
def test_f2_input_transform_bitexact(shape, layout):
    torch = torch_dev()
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(21, n, cin, cout, h, w, signed=True)
    eb = [int(v) for v in np.random.default_rng(22).integers(0, 4, 16)]
    gp = W.wino_f2_plan(f, eb, bias=b)
    ws = workspace(gp, n, h, w)
    th, tw = tapwise.tile_grid(h, w, 2)
    vq = torch.empty((16, n * th * tw, cin), dtype=torch.int8, device="cuda")
    W.wino_f4_debug_input_transform(gp, to_device(x, layout), n, h, w, layout, vq, ws)
    torch.cuda.synchronize()
    assert (vq.cpu().numpy() == tapwise.input_taps_quantized(x, eb, m=2)).all()


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", SHAPES)
def test_f2_tap_gemm_bitexact(shape, layout):
    torch = torch_dev()
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(23, n, cin, cout, h, w, signed=True)
    eb = [int(v) for v in np.random.default_rng(24).integers(0, 4, 16)]
    gp, op = _pair(f, eb, b, 0, False)
    ws = workspace(gp, n, h, w)
    th, tw = tapwise.tile_grid(h, w, 2)
    m = torch.empty((16, n * th * tw, cout), dtype=torch.int32, device="cuda")
    W.wino_f4_debug_tap_gemm(gp, to_device(x, layout), n, h, w, layout, m, ws)
    torch.cuda.synchronize()
    ref = tapwise.tap_gemm(tapwise.input_taps_quantized(x, eb, m=2), op["uq"])
    assert (m.cpu().numpy().astype(np.int64) == ref).all()


@pytest.mark.parametrize("variant", [W.SPLIT, W.FUSED])
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("relu,out_shift", [(False, 7), (True, 10), (False, 0)])
def test_f2_conv_bitexact_random(shape, layout, relu, out_shift, variant):
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(25, n, cin, cout, h, w, signed=True)
    eb = tapwise.calibrate_input_exps(x, m=2)
    gp, op = _pair(f, eb, b, out_shift, relu)
    assert W.wino_f4_plan_info(gp)["epilogue_bits"] == 32
    y = run_conv(gp, x, layout, variant)
    ref = tapwise.conv_int8(x, op)
    assert (y == ref).all(), f"{(y != ref).sum()} mismatches"


@pytest.mark.parametrize("variant", [W.SPLIT, W.FUSED])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_f2_conv_int64_epilogue(layout, variant):
    n, cin, cout, h, w = 1, 20, 24, 11, 10
    x, f, b = workloads.random_case(26, n, cin, cout, h, w, signed=True)
    eb = [0] * 16
    eb[15], eb[0] = 15, 14
    gp, op = _pair(f, eb, b, 20, False)
    assert W.wino_f4_plan_info(gp)["epilogue_bits"] == 64
    assert (run_conv(gp, x, layout, variant) == tapwise.conv_int8(x, op)).all()


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", [(1, 3, 5, 7, 9), (2, 64, 40, 16, 20), (1, 200, 8, 9, 9)])
def test_f2_calibrate_input_matches_oracle(shape, layout):
    torch_dev()
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(27, n, cin, cout, h, w, signed=True)
    eb, amax = W.wino_f2_calibrate_input(to_device(x, layout), n, cin, h, w, layout)
    assert amax == tapwise.input_tap_absmax(x, m=2)
    assert eb == tapwise.calibrate_input_exps(x, m=2)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_f2_calibrate_output_matches_oracle(layout):
    torch_dev()
    n, cin, cout, h, w = 2, 24, 40, 13, 18
    x, f, b = workloads.random_case(28, n, cin, cout, h, w, signed=False, zero_frac=0.3)
    eb = tapwise.calibrate_input_exps(x, m=2)
    gp, op = _pair(f, eb, b, 0, False)
    s, zmax = W.wino_f4_calibrate_output(gp, to_device(x, layout), n, h, w, layout, workspace(gp, n, h, w))
    z = tapwise.prequant_output(x, op)
    assert zmax == int(np.abs(z).max())
    assert s == tapwise.calibrate_out_shift(x, op)


def test_f2_i10_fused_is_unsupported():
    """The FUSED kernel has no 10-bit form; an int8/10 F2 plan is refused
    before any launch and the output is left alone."""
    torch = torch_dev()
    f = np.zeros((4, 4, 3, 3), np.float32)
    gp = W.wino_f2_plan_i10(f, [0] * 16)
    x = torch.zeros((1, 4, 8, 8), dtype=torch.int8, device="cuda")
    y = torch.full((1, 4, 8, 8), 7, dtype=torch.int8, device="cuda")
    with pytest.raises(W.WinoError) as e:
        W.wino_f4_conv_int8(gp, x, y, 1, 8, 8, W.NCHW, W.FUSED)
    assert e.value.status == -2
    torch.cuda.synchronize()
    assert (y.cpu().numpy() == 7).all()


def _config_layer(x, f, b, spec, layout, variant=W.SPLIT):
    """Calibrate (GPU) and run one layer with an F2 plan; returns GPU output
    and the oracle's for the same tables."""
    torch = torch_dev()
    n, cin, h, w = x.shape
    xd = to_device(x, layout)
    eb, _ = W.wino_f2_calibrate_input(xd, n, cin, h, w, layout)
    assert eb == tapwise.calibrate_input_exps(x, m=2)
    plan0 = W.wino_f2_plan(f, eb, bias=b, out_shift=0, relu=spec.relu)
    op0 = tapwise.make_plan(f, eb, bias=b, out_shift=0, relu=spec.relu, m=2)
    if spec.out_shift is None:
        s, _ = W.wino_f4_calibrate_output(plan0, xd, n, h, w, layout, workspace(plan0, n, h, w))
        assert s == tapwise.calibrate_out_shift(x, op0)
    else:
        s = spec.out_shift
    plan = W.wino_f2_plan(f, eb, bias=b, out_shift=s, relu=spec.relu)
    op = tapwise.make_plan(f, eb, bias=b, out_shift=s, relu=spec.relu, m=2)
    shape = (n, spec.cout, h, w) if layout == W.NCHW else (n, h, w, spec.cout)
    y = torch.full(shape, 77, dtype=torch.int8, device="cuda")
    ws = workspace(plan, n, h, w) if variant == W.SPLIT else None
    W.wino_f4_conv_int8(plan, xd, y, n, h, w, layout, variant, ws)
    torch.cuda.synchronize()
    return from_device_nchw(y, layout), tapwise.conv_int8(x, op)


@pytest.mark.parametrize("variant", [W.SPLIT, W.FUSED])
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("name", ["C1", "C2"])
def test_f2_config_bitexact(name, layout, variant):
    x, layers = workloads.generate(name)
    f, b, spec = layers[0]
    y, ref = _config_layer(x, f, b, spec, layout, variant)
    assert (y == ref).all()


@pytest.mark.parametrize("variant", [W.SPLIT, W.FUSED])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_f2_c3_chain_bitexact(layout, variant):
    """The four chained C3 layers with F2 plans, each fed the GPU's own
    previous output (max-pooled where the stage halves the image)."""
    x, layers = workloads.generate("C3")
    cur = x
    for k, (f, b, spec) in enumerate(layers):
        if k > 0:
            cur = workloads.next_layer_input(cur, spec)
        y, ref = _config_layer(cur, f, b, spec, layout, variant)
        assert (y == ref).all(), f"layer {k}"
        cur = y
