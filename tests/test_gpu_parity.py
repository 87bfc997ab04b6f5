"""GPU parity: the HIP path through the C ABI against the CPU oracle, bit for
bit (integer path: exact equality is the only correct result)."""
import numpy as np
import pytest

import paper_2209_12982_amd as W
import workloads
from oracle import direct, tapwise

from gpu_util import empty_out, from_device_nchw, run_conv, to_device, torch_dev, workspace

pytestmark = pytest.mark.gpu

LAYOUTS = [W.NCHW, W.NHWC]


def _plan_pair(f, eb, bias, out_shift, relu, e_g=None):
    gp = W.wino_f4_plan(f, eb, w_exp=e_g, bias=bias, out_shift=out_shift, relu=relu)
    op = tapwise.make_plan(f, eb, e_g=e_g, bias=bias, out_shift=out_shift, relu=relu)
    return gp, op


SHAPES = [
    # n, cin, cout, h, w
    (1, 1, 1, 1, 1),
    (1, 3, 5, 7, 9),
    (2, 16, 16, 8, 8),
    (1, 64, 64, 17, 13),
    (2, 70, 80, 12, 30),
    (1, 130, 33, 5, 66),
    (3, 8, 100, 2, 3),
]


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", SHAPES)
def test_input_transform_bitexact(shape, layout):
    torch = torch_dev()
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(1, n, cin, cout, h, w, signed=True)
    eb = [int(v) for v in np.random.default_rng(2).integers(0, 9, 36)]
    gp = W.wino_f4_plan(f, eb, bias=b)
    ws = workspace(gp, n, h, w)
    th, tw = tapwise.tile_grid(h, w)
    vq = torch.empty((36, n * th * tw, cin), dtype=torch.int8, device="cuda")
    W.wino_f4_debug_input_transform(gp, to_device(x, layout), n, h, w, layout, vq, ws)
    torch.cuda.synchronize()
    ref = tapwise.input_taps_quantized(x, eb)
    assert (vq.cpu().numpy() == ref).all()


# NHWC input-transform kernels: the direct kernel with 16-tile blocks (rows of
# 16 and 32 tiles, ragged image edges, several blocks per row) and 8-tile
# blocks, Cin % 4 == 0 but not % 16, and Cin % 4 != 0 (the LDS-band kernel)
K1_SHAPES = [
    # n, cin, h, w
    (1, 64, 9, 64),       # 16 tiles per row: one 16-tile block, ragged rows
    (2, 72, 5, 125),      # 32 tiles per row, last column ragged: two 16-tile blocks
    (1, 12, 7, 37),       # 10 tiles per row: 8-tile blocks, Cin % 16 != 0
    (1, 130, 6, 70),      # 18 tiles per row, Cin % 4 != 0: the LDS-band kernel
    (3, 4, 3, 3),         # one tile, four channels
]


@pytest.mark.parametrize("m", [4, 2])
@pytest.mark.parametrize("shape", K1_SHAPES)
def test_input_transform_nhwc_block_widths(shape, m):
    torch = torch_dev()
    n, cin, h, w = shape
    x, f, b = workloads.random_case(11, n, cin, 8, h, w, signed=True)
    ntap = (m + 2) ** 2
    eb = [int(v) for v in np.random.default_rng(12).integers(0, 9, ntap)]
    gp = (W.wino_f4_plan if m == 4 else W.wino_f2_plan)(f, eb, bias=b)
    ws = workspace(gp, n, h, w)
    th, tw = tapwise.tile_grid(h, w, m)
    vq = torch.empty((ntap, n * th * tw, cin), dtype=torch.int8, device="cuda")
    W.wino_f4_debug_input_transform(gp, to_device(x, W.NHWC), n, h, w, W.NHWC, vq, ws)
    torch.cuda.synchronize()
    ref = tapwise.input_taps_quantized(x, eb, m=m)
    assert (vq.cpu().numpy() == ref).all()


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", SHAPES)
def test_tap_gemm_bitexact(shape, layout):
    torch = torch_dev()
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(3, n, cin, cout, h, w, signed=True)
    eb = [int(v) for v in np.random.default_rng(4).integers(0, 9, 36)]
    gp, op = _plan_pair(f, eb, b, 0, False)
    ws = workspace(gp, n, h, w)
    th, tw = tapwise.tile_grid(h, w)
    m = torch.empty((36, n * th * tw, cout), dtype=torch.int32, device="cuda")
    W.wino_f4_debug_tap_gemm(gp, to_device(x, layout), n, h, w, layout, m, ws)
    torch.cuda.synchronize()
    ref = tapwise.tap_gemm(tapwise.input_taps_quantized(x, eb), op["uq"])
    assert (m.cpu().numpy().astype(np.int64) == ref).all()


VARIANTS = [W.SPLIT, W.FUSED]


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("relu,out_shift", [(False, 9), (True, 12)])
def test_conv_bitexact_random(shape, layout, relu, out_shift, variant):
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(5, n, cin, cout, h, w, signed=True)
    eb = tapwise.calibrate_input_exps(x)
    gp, op = _plan_pair(f, eb, b, out_shift, relu)
    assert W.wino_f4_plan_info(gp)["epilogue_bits"] == 32
    y = run_conv(gp, x, layout, variant)
    ref = tapwise.conv_int8(x, op)
    assert (y == ref).all(), f"{(y != ref).sum()} mismatches"


# shapes for the row-streamed tap GEMM: 1..5 k-chunks of 64 input channels,
# ragged tile counts and channel counts that leave partial 64-blocks
ROWS_SHAPES = SHAPES + [
    (1, 256, 200, 21, 26),
    (2, 192, 64, 9, 40),
    (1, 320, 128, 16, 16),
    (3, 128, 72, 14, 14),
]


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", ROWS_SHAPES)
@pytest.mark.parametrize("relu,out_shift", [(False, 9), (True, 12), (False, 0)])
def test_conv_rows_kernel_bitexact(shape, layout, relu, out_shift):
    """The row-streamed tap GEMM, forced on shapes the automatic choice
    would give to the tap-resident kernel."""
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(5, n, cin, cout, h, w, signed=True)
    eb = tapwise.calibrate_input_exps(x)
    gp, op = _plan_pair(f, eb, b, out_shift, relu)
    W.wino_f4_plan_set_tap_kernel(gp, W.TAP_ROWS)
    y = run_conv(gp, x, layout, W.SPLIT)
    ref = tapwise.conv_int8(x, op)
    assert (y == ref).all(), f"{(y != ref).sum()} mismatches"


# shapes for the wave-specialized tap GEMM: ring stages of 1..4 k-chunks
# (input channels 64, 128, 192, 256 padded), several stages per tap (320:
# five one-chunk stages, 512: two four-chunk stages), ragged tiles and
# channel counts that leave partial 64-blocks, images smaller than a tile
WAVES_SHAPES = SHAPES + [
    (1, 256, 200, 21, 26),
    (2, 192, 64, 9, 40),
    (1, 320, 128, 16, 16),
    (3, 128, 72, 14, 14),
    (1, 512, 64, 12, 20),
    (2, 64, 130, 3, 2),
    (1, 33, 256, 40, 8),
]


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", WAVES_SHAPES)
@pytest.mark.parametrize("relu,out_shift", [(False, 9), (True, 12), (False, 0)])
def test_conv_waves_kernel_bitexact(shape, layout, relu, out_shift):
    """The wave-specialized tap GEMM (MFMA waves + fold waves), forced on
    every shape."""
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(7, n, cin, cout, h, w, signed=True)
    eb = tapwise.calibrate_input_exps(x)
    gp, op = _plan_pair(f, eb, b, out_shift, relu)
    W.wino_f4_plan_set_tap_kernel(gp, W.TAP_WAVES)
    assert W.wino_f4_tap_kernel_choice(gp, n, h, w) == W.TAP_WAVES
    y = run_conv(gp, x, layout, W.SPLIT)
    ref = tapwise.conv_int8(x, op)
    assert (y == ref).all(), f"{(y != ref).sum()} mismatches"


def test_tap_kernel_choice():
    torch_dev()
    f = np.random.default_rng(9).normal(0, 0.05, (256, 256, 3, 3)).astype(np.float32)
    plan = W.wino_f4_plan(f, [4] * 36, bias=None, out_shift=11)
    # 4 x 160 x 160: 400 blocks of 64 x 64 fill the device; 1 x 56 x 56: 4 do not
    assert W.wino_f4_tap_kernel_choice(plan, 4, 160, 160) == W.TAP_ROWS
    assert W.wino_f4_tap_kernel_choice(plan, 1, 56, 56) == W.TAP_RESIDENT_64X32
    W.wino_f4_plan_set_tap_kernel(plan, W.TAP_RESIDENT)
    assert W.wino_f4_tap_kernel_choice(plan, 4, 160, 160) == W.TAP_RESIDENT_64X32
    W.wino_f4_plan_set_tap_kernel(plan, W.TAP_ROWS)
    assert W.wino_f4_tap_kernel_choice(plan, 1, 56, 56) == W.TAP_ROWS
    assert W.wino_f4_tap_kernel_choice(plan, 4, 160, 160) == W.TAP_ROWS
    W.wino_f4_plan_set_tap_kernel(plan, W.TAP_WAVES)
    assert W.wino_f4_tap_kernel_choice(plan, 1, 56, 56) == W.TAP_WAVES
    for kind in (W.TAP_RESIDENT_64X32, W.TAP_RESIDENT_32X32, W.TAP_RESIDENT_16X16):
        W.wino_f4_plan_set_tap_kernel(plan, kind)
        assert W.wino_f4_tap_kernel_choice(plan, 4, 160, 160) == kind
    with pytest.raises(W.WinoError):
        W.wino_f4_tap_kernel_choice(plan, -1, 8, 8)
    # the 64-bit epilogue always runs the tap-resident kernel
    eb = [0] * 36
    eb[35], eb[0] = 15, 14
    p64 = W.wino_f4_plan(f[:24, :20], eb, bias=None, out_shift=20)
    assert W.wino_f4_plan_info(p64)["epilogue_bits"] == 64
    for kind in (W.TAP_ROWS, W.TAP_WAVES):
        W.wino_f4_plan_set_tap_kernel(p64, kind)
        assert W.wino_f4_tap_kernel_choice(p64, 4, 160, 160) == W.TAP_RESIDENT_64X32


@pytest.mark.parametrize("kind", [W.TAP_RESIDENT_32X32, W.TAP_RESIDENT_16X16])
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", SHAPES + [(1, 256, 200, 21, 26), (2, 192, 48, 9, 40)])
@pytest.mark.parametrize("relu,out_shift", [(False, 9), (True, 0)])
def test_conv_resident_shapes_bitexact(shape, layout, relu, out_shift, kind):
    """The small-layer block shapes of the tap-resident kernel, forced."""
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(5, n, cin, cout, h, w, signed=True)
    eb = tapwise.calibrate_input_exps(x)
    gp, op = _plan_pair(f, eb, b, out_shift, relu)
    W.wino_f4_plan_set_tap_kernel(gp, kind)
    y = run_conv(gp, x, layout, W.SPLIT)
    ref = tapwise.conv_int8(x, op)
    assert (y == ref).all(), f"{(y != ref).sum()} mismatches"


@pytest.mark.parametrize("kind", [W.TAP_RESIDENT_32X32, W.TAP_RESIDENT_16X16])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_conv_resident_shapes_int64(layout, kind):
    n, cin, cout, h, w = 1, 20, 24, 11, 10
    x, f, b = workloads.random_case(6, n, cin, cout, h, w, signed=True)
    eb = [0] * 36
    eb[35], eb[0] = 15, 14
    gp, op = _plan_pair(f, eb, b, 20, False)
    assert W.wino_f4_plan_info(gp)["epilogue_bits"] == 64
    W.wino_f4_plan_set_tap_kernel(gp, kind)
    assert (run_conv(gp, x, layout, W.SPLIT) == tapwise.conv_int8(x, op)).all()


@pytest.mark.parametrize("layout", LAYOUTS)
def test_tap_kernels_agree(layout):
    """Both tap-GEMM kernels on one plan, two calls each, equal to the oracle."""
    n, cin, cout, h, w = 2, 128, 128, 40, 36
    x, f, b = workloads.random_case(8, n, cin, cout, h, w, signed=False, zero_frac=0.5)
    eb = tapwise.calibrate_input_exps(x)
    gp, op = _plan_pair(f, eb, b, 11, False)
    ref = tapwise.conv_int8(x, op)
    for kind in (W.TAP_ROWS, W.TAP_RESIDENT, W.TAP_RESIDENT_16X16, W.TAP_ROWS, W.TAP_RESIDENT_32X32,
                 W.TAP_RESIDENT_64X32, W.TAP_AUTO):
        W.wino_f4_plan_set_tap_kernel(gp, kind)
        assert (run_conv(gp, x, layout, W.SPLIT) == ref).all(), f"tap kernel {kind}"


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("layout", LAYOUTS)
def test_fused_equals_split_unaligned_channels(layout, variant):
    """Odd channel counts exercise the byte-wise loads of both variants."""
    n, cin, cout, h, w = 1, 67, 33, 10, 13
    x, f, b = workloads.random_case(11, n, cin, cout, h, w, signed=True)
    eb = tapwise.calibrate_input_exps(x)
    gp, op = _plan_pair(f, eb, b, 10, False)
    assert (run_conv(gp, x, layout, variant) == tapwise.conv_int8(x, op)).all()


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("layout", LAYOUTS)
def test_conv_int64_epilogue(layout, variant):
    """Large alignment shifts force the 64-bit output transform."""
    n, cin, cout, h, w = 1, 20, 24, 11, 10
    x, f, b = workloads.random_case(6, n, cin, cout, h, w, signed=True)
    eb = [0] * 36
    eb[35] = 15
    eb[0] = 14
    gp, op = _plan_pair(f, eb, b, 20, False)
    assert W.wino_f4_plan_info(gp)["epilogue_bits"] == 64
    y = run_conv(gp, x, layout, variant)
    assert (y == tapwise.conv_int8(x, op)).all()


@pytest.mark.parametrize("variant", VARIANTS)
def test_conv_deterministic_repeat(variant):
    n, cin, cout, h, w = 2, 96, 96, 30, 30
    x, f, b = workloads.random_case(7, n, cin, cout, h, w, signed=False, zero_frac=0.5)
    eb = tapwise.calibrate_input_exps(x)
    gp = W.wino_f4_plan(f, eb, bias=b, out_shift=11)
    y1 = run_conv(gp, x, W.NHWC, variant)
    y2 = run_conv(gp, x, W.NHWC, variant)
    assert (y1 == y2).all()


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", [(1, 3, 5, 7, 9), (2, 64, 40, 16, 20), (1, 200, 8, 9, 9)])
def test_calibrate_input_matches_oracle(shape, layout):
    torch_dev()
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(8, n, cin, cout, h, w, signed=True)
    eb, amax = W.wino_f4_calibrate_input(to_device(x, layout), n, cin, h, w, layout)
    assert amax == tapwise.input_tap_absmax(x)
    assert eb == tapwise.calibrate_input_exps(x)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_calibrate_output_matches_oracle(layout):
    torch_dev()
    n, cin, cout, h, w = 2, 24, 40, 13, 18
    x, f, b = workloads.random_case(9, n, cin, cout, h, w, signed=False, zero_frac=0.3)
    eb = tapwise.calibrate_input_exps(x)
    gp, op = _plan_pair(f, eb, b, 0, False)
    s, zmax = W.wino_f4_calibrate_output(gp, to_device(x, layout), n, h, w, layout, workspace(gp, n, h, w))
    z = tapwise.prequant_output(x, op)
    assert zmax == int(np.abs(z).max())
    assert s == tapwise.calibrate_out_shift(x, op)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape", [(1, 16, 16, 32, 32), (2, 3, 5, 7, 9), (1, 70, 130, 9, 14),
                                   (2, 64, 130, 9, 14), (1, 128, 64, 17, 23), (3, 192, 40, 5, 7),
                                   (1, 64, 256, 1, 1), (2, 256, 128, 16, 16), (1, 64, 320, 19, 70),
                                   (2, 128, 96, 33, 40), (1, 64, 8, 8, 32), (1, 64, 72, 13, 36),
                                   (2, 64, 40, 7, 4), (1, 64, 300, 9, 20)])
def test_direct_conv_bitexact(shape, layout):
    torch = torch_dev()
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(10, n, cin, cout, h, w, signed=True)
    w_ohwi, e = W.direct_conv_quantize_weights(f)
    wq_ref, e_ref = direct.quantize_weights_pow2(f)
    assert e == e_ref and (w_ohwi == wq_ref.transpose(0, 2, 3, 1)).all()
    y = empty_out(n, cout, h, w, layout)
    W.direct_conv_int8(to_device(x, layout), torch.from_numpy(w_ohwi).cuda(), torch.from_numpy(b).cuda(), y,
                       n, cin, cout, h, w, layout, 9, False)
    torch.cuda.synchronize()
    ref = direct.conv_int8(x, wq_ref, b, 9, False)
    assert (from_device_nchw(y, layout) == ref).all()


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("shape,relu,shift,with_bias", [
    ((1, 64, 3, 9, 8), True, 0, True),          # three output channels, no shift
    ((2, 128, 260, 5, 12), False, 14, False),   # no bias, a partial second channel block
    ((1, 64, 64, 1, 4), True, 7, True),         # one output row, one four-pixel column group
    ((3, 64, 32, 17, 64), False, 9, True),      # two tile columns, three images
])
def test_direct_conv_options(shape, relu, shift, with_bias, layout):
    """The tile kernel's options and edges: ReLU, out_shift 0, a NULL bias,
    Cout below four, a partial channel block, single rows and narrow images."""
    torch = torch_dev()
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(14, n, cin, cout, h, w, signed=True)
    w_ohwi, _ = W.direct_conv_quantize_weights(f)
    wq_ref, _ = direct.quantize_weights_pow2(f)
    y = empty_out(n, cout, h, w, layout)
    bd = torch.from_numpy(b).cuda() if with_bias else None
    W.direct_conv_int8(to_device(x, layout), torch.from_numpy(w_ohwi).cuda(), bd, y, n, cin, cout, h, w, layout,
                       shift, relu)
    torch.cuda.synchronize()
    ref = direct.conv_int8(x, wq_ref, b if with_bias else None, shift, relu)
    assert (from_device_nchw(y, layout) == ref).all()


@pytest.mark.parametrize("layout", LAYOUTS)
def test_direct_conv_wide_bias(layout):
    """Biases near the int32 limits: acc + bias + rounding leaves int32 for
    some channels, so the requantization must widen (the fast path keeps 32
    bits only when every bias of a channel block leaves room); out_shift 31."""
    torch = torch_dev()
    n, cin, cout, h, w = 1, 64, 80, 11, 16
    x, f, _ = workloads.random_case(12, n, cin, cout, h, w, signed=True)
    b = np.random.default_rng(13).integers(-2 ** 31, 2 ** 31, cout).astype(np.int64)
    b[::3] = 2 ** 31 - 1
    b[1::3] = -2 ** 31
    b = b.astype(np.int32)
    w_ohwi, e = W.direct_conv_quantize_weights(f)
    wq_ref, _ = direct.quantize_weights_pow2(f)
    for shift in (31, 20):
        y = empty_out(n, cout, h, w, layout)
        W.direct_conv_int8(to_device(x, layout), torch.from_numpy(w_ohwi).cuda(), torch.from_numpy(b).cuda(), y,
                           n, cin, cout, h, w, layout, shift, False)
        torch.cuda.synchronize()
        assert (from_device_nchw(y, layout) == direct.conv_int8(x, wq_ref, b, shift, False)).all(), shift


@pytest.mark.parametrize("layout", LAYOUTS)
def test_config_c1_bitexact(layout):
    """C1 as specified: out_shift 8 (the literal value), calibrated e_B."""
    x, layers = workloads.generate("C1")
    f, b, spec = layers[0]
    eb_gpu, _ = W.wino_f4_calibrate_input(to_device(x, layout), *[x.shape[0], spec.cin, spec.h, spec.w], layout)
    eb = tapwise.calibrate_input_exps(x)
    assert eb_gpu == eb
    gp, op = _plan_pair(f, eb, b, 8, False)
    y = run_conv(gp, x, layout)
    assert (y == tapwise.conv_int8(x, op)).all()


@pytest.mark.parametrize("layout", LAYOUTS)
def test_config_c1_calibrated_shift_bitexact(layout):
    """C1 with the output shift calibrated like C2-C5 (max |Y + bias| on the
    layer's own input) instead of the literal 8: the GPU's calibration must
    pick the oracle's shift and the layer must match byte for byte."""
    x, layers = workloads.generate("C1")
    f, b, spec = layers[0]
    n = x.shape[0]
    xd = to_device(x, layout)
    eb, _ = W.wino_f4_calibrate_input(xd, n, spec.cin, spec.h, spec.w, layout)
    assert eb == tapwise.calibrate_input_exps(x)
    gp0 = W.wino_f4_plan(f, eb, bias=b)
    s, _ = W.wino_f4_calibrate_output(gp0, xd, n, spec.h, spec.w, layout, workspace(gp0, n, spec.h, spec.w))
    s_ref = tapwise.calibrate_out_shift(x, tapwise.make_plan(f, eb, bias=b, out_shift=0))
    assert s == s_ref and s != 8
    gp, op = _plan_pair(f, eb, b, s, False)
    y = run_conv(gp, x, layout)
    assert (y == tapwise.conv_int8(x, op)).all()


def test_tap_gemm_export_full_channels():
    """The raw tap-GEMM result M (no output transform) on one image of the
    C5 layer, all 256 -> 256 channels: every int32 of the 36 x 1600 x 256
    export against the oracle's tap-major GEMM."""
    torch = torch_dev()
    x, layers = workloads.generate("C5")
    f, b, spec = layers[0]
    x1 = np.ascontiguousarray(x[:1])
    eb = tapwise.calibrate_input_exps(x1)
    gp, op = _plan_pair(f, eb, b, 0, False)
    h, w = spec.h, spec.w
    th, tw = tapwise.tile_grid(h, w)
    m = torch.empty((36, th * tw, spec.cout), dtype=torch.int32, device="cuda")
    W.wino_f4_debug_tap_gemm(gp, to_device(x1, W.NHWC), 1, h, w, W.NHWC, m, workspace(gp, 1, h, w))
    torch.cuda.synchronize()
    ref = tapwise.tap_gemm(tapwise.input_taps_quantized(x1, eb), op["uq"])
    assert (m.cpu().numpy().astype(np.int64) == ref).all()


@pytest.mark.parametrize("layout", LAYOUTS)
def test_config_c2_bitexact(layout):
    x, layers = workloads.generate("C2")
    f, b, spec = layers[0]
    n = x.shape[0]
    xd = to_device(x, layout)
    eb, _ = W.wino_f4_calibrate_input(xd, n, spec.cin, spec.h, spec.w, layout)
    assert eb == tapwise.calibrate_input_exps(x)
    gp0 = W.wino_f4_plan(f, eb, bias=b)
    s, _ = W.wino_f4_calibrate_output(gp0, xd, n, spec.h, spec.w, layout, workspace(gp0, n, spec.h, spec.w))
    op = tapwise.make_plan(f, eb, bias=b, out_shift=0)
    assert s == tapwise.calibrate_out_shift(x, op)
    gp, op = _plan_pair(f, eb, b, s, False)
    y = run_conv(gp, x, layout)
    assert (y == tapwise.conv_int8(x, op)).all()
