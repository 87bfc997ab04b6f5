"""GPU parity of the int8/10 variant (10-bit Winograd-domain integers, Sec. V;
plans from wino_f4_plan_i10 / wino_f2_plan_i10) through the C ABI against
the oracle's 10-bit pipeline, bit for bit: the fp16 Winograd-domain input,
the tap GEMM, whole convolutions on ragged shapes, both epilogue widths,
calibration, and the full-size configurations (oracle results stored in
tests/golden/configs_i10.json by tests/golden/make_golden.py --bits 10)."""
import hashlib
import json
import os

import numpy as np
import pytest

import paper_2209_12982_amd as W
import workloads
from oracle import direct, tapwise

from gpu_util import from_device_nchw, run_conv, to_device, torch_dev, workspace

pytestmark = pytest.mark.gpu

LAYOUTS = [W.NCHW, W.NHWC]
MS = [4, 2]
SHAPES = [
    # n, cin, cout, h, w
    (1, 1, 1, 1, 1),
    (1, 3, 5, 7, 9),
    (2, 16, 16, 8, 8),
    (1, 64, 64, 17, 13),
    (2, 70, 80, 12, 30),
    (1, 130, 33, 5, 66),
    (1, 256, 64, 14, 14),
]
GOLDEN_PATH = os.path.join(os.path.dirname(__file__), "golden", "configs_i10.json")


def _ntap(m):
    return (m + 2) ** 2


def _plan(m, f, eb, **kw):
    return (W.wino_f4_plan_i10 if m == 4 else W.wino_f2_plan_i10)(f, eb, **kw)


def _calibrate(m, xd, n, cin, h, w, layout):
    return (W.wino_f4_calibrate_input_i10 if m == 4 else W.wino_f2_calibrate_input_i10)(xd, n, cin, h, w, layout)


def _oplan(m, f, eb, **kw):
    return tapwise.make_plan(f, eb, m=m, bits=10, **kw)


@pytest.mark.parametrize("m", MS)
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", SHAPES)
def test_i10_input_transform_bitexact(m, shape, layout):
    torch = torch_dev()
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(51, n, cin, cout, h, w, signed=True)
    # small exponents drive many taps to the 10-bit rails
    eb = [int(v) for v in np.random.default_rng(52).integers(0, 5, _ntap(m))]
    gp = _plan(m, f, eb, bias=b)
    ws = workspace(gp, n, h, w)
    th, tw = tapwise.tile_grid(h, w, m)
    vq = torch.empty((_ntap(m), n * th * tw, cin), dtype=torch.float16, device="cuda")
    W.wino_f4_debug_input_transform(gp, to_device(x, layout), n, h, w, layout, vq, ws)
    torch.cuda.synchronize()
    got = vq.cpu().numpy().astype(np.int64)
    ref = tapwise.input_taps_quantized(x, eb, m=m, bits=10)
    assert (got == ref).all(), f"{(got != ref).sum()} mismatches"
    assert np.abs(ref).max() > 127 or n * h * w < 64        # the 10-bit range is in use


@pytest.mark.parametrize("m", MS)
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", SHAPES)
def test_i10_tap_gemm_bitexact(m, shape, layout):
    torch = torch_dev()
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(53, n, cin, cout, h, w, signed=True)
    eb = [int(v) for v in np.random.default_rng(54).integers(0, 5, _ntap(m))]
    gp = _plan(m, f, eb, bias=b)
    op = _oplan(m, f, eb, bias=b)
    ws = workspace(gp, n, h, w)
    th, tw = tapwise.tile_grid(h, w, m)
    mm = torch.empty((_ntap(m), n * th * tw, cout), dtype=torch.int32, device="cuda")
    W.wino_f4_debug_tap_gemm(gp, to_device(x, layout), n, h, w, layout, mm, ws)
    torch.cuda.synchronize()
    ref = tapwise.tap_gemm(tapwise.input_taps_quantized(x, eb, m=m, bits=10), op["uq"])
    assert (mm.cpu().numpy().astype(np.int64) == ref).all()


@pytest.mark.parametrize("m", MS)
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("relu,out_shift", [(False, 9), (True, 12), (False, 0)])
def test_i10_conv_bitexact_random(m, shape, layout, relu, out_shift):
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(55, n, cin, cout, h, w, signed=True)
    eb = tapwise.calibrate_input_exps(x, m=m, bits=10)
    gp = _plan(m, f, eb, bias=b, out_shift=out_shift, relu=relu)
    op = _oplan(m, f, eb, bias=b, out_shift=out_shift, relu=relu)
    y = run_conv(gp, x, layout)
    ref = tapwise.conv_int8(x, op)
    assert (y == ref).all(), f"{(y != ref).sum()} mismatches"


@pytest.mark.parametrize("m", MS)
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("bits_wanted", [32, 64])
def test_i10_conv_both_epilogues(m, layout, bits_wanted):
    """Small input exponents keep the 32-bit epilogue; unequal large ones
    (wide alignment shifts) force the 64-bit one."""
    n, cin, cout, h, w = 1, 40, 72, 11, 14
    x, f, b = workloads.random_case(56, n, cin, cout, h, w, signed=True)
    eb = [0] * _ntap(m) if bits_wanted == 32 else [15 if t % 3 == 0 else 0 for t in range(_ntap(m))]
    f = f * (0.05 if bits_wanted == 32 else 1.0)
    gp = _plan(m, f, eb, bias=b, out_shift=16)
    op = _oplan(m, f, eb, bias=b, out_shift=16)
    assert W.wino_f4_plan_info(gp)["epilogue_bits"] == bits_wanted
    assert (run_conv(gp, x, layout) == tapwise.conv_int8(x, op)).all()


@pytest.mark.parametrize("m", MS)
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", [(1, 3, 5, 7, 9), (2, 64, 40, 16, 20), (1, 200, 8, 9, 9)])
def test_i10_calibrate_input_matches_oracle(m, shape, layout):
    torch_dev()
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(57, n, cin, cout, h, w, signed=True)
    eb, amax = _calibrate(m, to_device(x, layout), n, cin, h, w, layout)
    assert amax == tapwise.input_tap_absmax(x, m=m)
    assert eb == tapwise.calibrate_input_exps(x, m=m, bits=10)


@pytest.mark.parametrize("m", MS)
@pytest.mark.parametrize("layout", LAYOUTS)
def test_i10_calibrate_output_matches_oracle(m, layout):
    torch_dev()
    n, cin, cout, h, w = 2, 24, 40, 13, 18
    x, f, b = workloads.random_case(58, n, cin, cout, h, w, signed=False, zero_frac=0.3)
    eb = tapwise.calibrate_input_exps(x, m=m, bits=10)
    gp = _plan(m, f, eb, bias=b)
    op = _oplan(m, f, eb, bias=b)
    s, zmax = W.wino_f4_calibrate_output(gp, to_device(x, layout), n, h, w, layout, workspace(gp, n, h, w))
    assert zmax == int(np.abs(tapwise.prequant_output(x, op)).max())
    assert s == tapwise.calibrate_out_shift(x, op)


def test_i10_unsupported_and_rejected_calls():
    torch = torch_dev()
    f = np.zeros((4, 4, 3, 3), np.float32)
    gp = W.wino_f4_plan_i10(f, [0] * 36)
    x = torch.zeros((1, 4, 8, 8), dtype=torch.int8, device="cuda")
    y = torch.zeros((1, 4, 8, 8), dtype=torch.int8, device="cuda")
    with pytest.raises(W.WinoError) as e:
        W.wino_f4_conv_int8(gp, x, y, 1, 8, 8, W.NCHW, W.FUSED)
    assert e.value.status == -2
    with pytest.raises(W.WinoError) as e:
        W.wino_f4_plan_info(gp, with_uq=True)
    assert e.value.status == -1
    # twice the 8-bit workspace: Vq is fp16
    g8 = W.wino_f4_plan(f, [0] * 36)
    assert W.wino_f4_workspace_bytes(gp, 2, 30, 30) == 2 * W.wino_f4_workspace_bytes(g8, 2, 30, 30)


def test_i10_tap_kernel_choice_and_forced_shapes():
    """int8/10 runs the row-streamed kernel with fp16 operands by default,
    with either epilogue width; RESIDENT picks the tap-resident 64x32 shape,
    or 32x32 with the 64-bit epilogue; a forced resident shape is honoured
    (16X16 stands for 32x32 blocks with 6-tap stages); every choice is
    exact.  Two k rows, 100 tiles in four blocks with a ragged last one."""
    n, cin, cout, h, w = 1, 64, 64, 40, 40
    x, f, b = workloads.random_case(59, n, cin, cout, h, w, signed=True)
    for eb, resident in (([0] * 36, W.TAP_RESIDENT_64X32),
                         ([15 if t % 3 == 0 else 0 for t in range(36)], W.TAP_RESIDENT_32X32)):
        f2 = f * (0.05 if resident == W.TAP_RESIDENT_64X32 else 1.0)
        gp = W.wino_f4_plan_i10(f2, eb, bias=b, out_shift=14)
        assert W.wino_f4_plan_info(gp)["epilogue_bits"] == (32 if resident == W.TAP_RESIDENT_64X32 else 64)
        op = _oplan(4, f2, eb, bias=b, out_shift=14)
        ref = tapwise.conv_int8(x, op)
        for forced, want in ((W.TAP_AUTO, W.TAP_ROWS), (W.TAP_ROWS, W.TAP_ROWS), (W.TAP_RESIDENT, resident),
                             (W.TAP_RESIDENT_64X32, W.TAP_RESIDENT_64X32),
                             (W.TAP_RESIDENT_32X32, W.TAP_RESIDENT_32X32),
                             (W.TAP_RESIDENT_16X16, W.TAP_RESIDENT_16X16)):
            W.wino_f4_plan_set_tap_kernel(gp, forced)
            assert W.wino_f4_tap_kernel_choice(gp, n, h, w) == want
            for layout in LAYOUTS:
                assert (run_conv(gp, x, layout) == ref).all(), (forced, layout)


def _config_layer(m, x, f, b, spec, layout):
    """Calibrate (GPU) and run one layer with a 10-bit plan; returns the GPU
    output and the oracle's for the same tables."""
    torch = torch_dev()
    n, cin, h, w = x.shape
    xd = to_device(x, layout)
    eb, _ = _calibrate(m, xd, n, cin, h, w, layout)
    assert eb == tapwise.calibrate_input_exps(x, m=m, bits=10)
    plan0 = _plan(m, f, eb, bias=b, out_shift=0, relu=spec.relu)
    op0 = _oplan(m, f, eb, bias=b, out_shift=0, relu=spec.relu)
    if spec.out_shift is None:
        s, _ = W.wino_f4_calibrate_output(plan0, xd, n, h, w, layout, workspace(plan0, n, h, w))
        assert s == tapwise.calibrate_out_shift(x, op0)
    else:
        s = spec.out_shift
    plan = _plan(m, f, eb, bias=b, out_shift=s, relu=spec.relu)
    op = _oplan(m, f, eb, bias=b, out_shift=s, relu=spec.relu)
    shape = (n, spec.cout, h, w) if layout == W.NCHW else (n, h, w, spec.cout)
    y = torch.full(shape, 77, dtype=torch.int8, device="cuda")
    W.wino_f4_conv_int8(plan, xd, y, n, h, w, layout, W.SPLIT, workspace(plan, n, h, w))
    torch.cuda.synchronize()
    return from_device_nchw(y, layout), tapwise.conv_int8(x, op)


@pytest.mark.parametrize("m", MS)
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("name", ["C1", "C2"])
def test_i10_config_bitexact(m, name, layout):
    x, layers = workloads.generate(name)
    f, b, spec = layers[0]
    y, ref = _config_layer(m, x, f, b, spec, layout)
    assert (y == ref).all()


@pytest.mark.parametrize("layout", LAYOUTS)
def test_i10_f2_c3_chain_bitexact(layout):
    x, layers = workloads.generate("C3")
    cur = x
    for k, (f, b, spec) in enumerate(layers):
        if k > 0:
            cur = workloads.next_layer_input(cur, spec)
        y, ref = _config_layer(2, cur, f, b, spec, layout)
        assert (y == ref).all(), f"layer {k}"
        cur = y


def _golden():
    if not os.path.exists(GOLDEN_PATH):
        pytest.skip("tests/golden/configs_i10.json not generated")
    return json.load(open(GOLDEN_PATH))


def _run_golden_layer(x, f, b, spec, rec, layout):
    torch = torch_dev()
    n, cin, h, w = x.shape
    xd = to_device(x, layout)
    eb, _ = W.wino_f4_calibrate_input_i10(xd, n, cin, h, w, layout)
    assert eb == rec["e_b"]
    plan0 = W.wino_f4_plan_i10(f, eb, bias=b, out_shift=0, relu=spec.relu)
    info0 = W.wino_f4_plan_info(plan0)
    assert info0["e_g"] == rec["e_g"] and info0["sh"] == rec["sh"] and info0["e_o"] == rec["e_o"]
    if spec.out_shift is None:
        s, zmax = W.wino_f4_calibrate_output(plan0, xd, n, h, w, layout, workspace(plan0, n, h, w))
        assert zmax == rec["zmax"] and s == rec["out_shift"]
    else:
        s = spec.out_shift
    plan = W.wino_f4_plan_i10(f, eb, bias=b, out_shift=s, relu=spec.relu)
    shape = (n, spec.cout, h, w) if layout == W.NCHW else (n, h, w, spec.cout)
    y = torch.full(shape, 77, dtype=torch.int8, device="cuda")
    W.wino_f4_conv_int8(plan, xd, y, n, h, w, layout, W.SPLIT, workspace(plan, n, h, w))
    torch.cuda.synchronize()
    yn = from_device_nchw(y, layout)
    for idx, v in rec["samples"]:
        assert int(yn[tuple(idx)]) == v, f"sample {idx}: {int(yn[tuple(idx)])} != {v}"
    assert hashlib.sha256(yn.tobytes()).hexdigest() == rec["sha256_nchw"]
    return yn


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("name", ["C4", "C5"])
def test_i10_full_size_layer_bitexact(name, layout):
    g = _golden()
    x, layers = workloads.generate(name)
    f, b, spec = layers[0]
    _run_golden_layer(x, f, b, spec, g[name]["layers"][0], layout)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_i10_c3_chain_full_size_bitexact(layout):
    g = _golden()
    x, layers = workloads.generate("C3")
    cur = x
    for k, (f, b, spec) in enumerate(layers):
        if k > 0:
            cur = workloads.next_layer_input(cur, spec)
        cur = _run_golden_layer(cur, f, b, spec, g["C3"]["layers"][k], layout)


def test_i10_is_more_accurate_than_int8():
    """What the variant is for: on a C2 layer, the 10-bit Winograd domain
    brings the dequantized output closer to the float convolution than the
    8-bit one (both computed on the GPU, before output requantization)."""
    torch = torch_dev()
    x, layers = workloads.generate("C2")
    f, b, spec = layers[0]
    n, cin, h, w = x.shape
    xd = to_device(x, W.NCHW)
    ref = direct.conv_f64(x, f.astype(np.float64))
    errs = {}
    for bits in (8, 10):
        cal = W.wino_f4_calibrate_input if bits == 8 else W.wino_f4_calibrate_input_i10
        mk = W.wino_f4_plan if bits == 8 else W.wino_f4_plan_i10
        eb, _ = cal(xd, n, cin, h, w, W.NCHW)
        gp = mk(f, eb)
        th, tw = tapwise.tile_grid(h, w, 4)
        mm = torch.empty((36, n * th * tw, spec.cout), dtype=torch.int32, device="cuda")
        W.wino_f4_debug_tap_gemm(gp, xd, n, h, w, W.NCHW, mm, workspace(gp, n, h, w))
        torch.cuda.synchronize()
        info = W.wino_f4_plan_info(gp)
        y = tapwise.assemble(tapwise.output_transform(mm.cpu().numpy().astype(np.int64), info["sh"]), n, h, w)
        errs[bits] = np.sqrt(np.mean((y * 2.0 ** info["e_o"] - ref) ** 2))
    assert errs[10] < 0.5 * errs[8]
