"""GPU parity of the tap GEMM's stream-K split (WINO_TAP_ROWS_STREAMK): the
row-streamed kernel with the stages of its last, partial round of blocks
spread over every compute unit, the pieces' partial sums exchanged through
the workspace and added by the last piece of each block to arrive.  Forced on
layers below one round of blocks, every block is split, into pieces as short
as one stage; the result must be the oracle's bytes.  A second launch on the
same workspace checks that each launch leaves its counters at zero, and a
workspace without the split's part runs the unsplit kernel with the same
result.  The full-size split (C5's 400 blocks: one whole round, then 144
blocks over all compute units) is checked against the golden digest in both
layouts by test_gpu_configs.py."""
import numpy as np
import pytest

import paper_2209_12982_amd as W
import workloads
from oracle import tapwise

from gpu_util import empty_out, from_device_nchw, to_device, torch_dev

pytestmark = pytest.mark.gpu

SHAPES = [
    # n, cin, cout, h, w      split blocks x stages per block -> stream-K workgroups
    (1, 64, 64, 20, 20),      # 1 x 6: six one-stage pieces of one block
    (2, 130, 70, 33, 18),     # 4 x 18, ragged channels and tiles: one stage each
    (1, 200, 40, 61, 43),     # 3 x 24: one stage each, a partial channel block
    (2, 256, 128, 64, 64),    # 16 x 24 over all compute units: ranges of 1-2 stages across block edges
    (1, 384, 64, 100, 100),   # 10 x 36: ranges of about 1.4 stages, six rows of taps each
]


def _ncu():
    return torch_dev().cuda.get_device_properties(0).multi_processor_count


def _plans(shape, seed, relu, out_shift=9):
    n, cin, cout, h, w = shape
    x, f, b = workloads.random_case(seed, n, cin, cout, h, w, signed=True)
    eb = tapwise.calibrate_input_exps(x)
    gp = W.wino_f4_plan(f, eb, bias=b, out_shift=out_shift, relu=relu)
    op = tapwise.make_plan(f, eb, bias=b, out_shift=out_shift, relu=relu)
    return x, gp, op


def _split_bytes(shape):
    # Vq, then the counters (one per split block) and two 256 KiB partial-sum
    # slots per stream-K workgroup, each part 256-byte aligned
    n, cin, cout, h, w = shape
    tiles = n * -(-h // 4) * -(-w // 4)
    vq = 36 * -(-tiles // 64) * 64 * -(-cin // 64) * 64
    blocks = -(-cout // 64) * -(-tiles // 64)
    split = blocks % _ncu()
    units = split * 6 * -(-cin // 64)
    groups = min(_ncu(), units)
    up = lambda v: -(-v // 256) * 256
    return vq, up(vq) + up(4 * split) + 2 * groups * 1024 * 64 * 4


def _conv(gp, x, layout, ws):
    torch = torch_dev()
    n, _, h, w = x.shape
    y = empty_out(n, gp.cout, h, w, layout)
    W.wino_f4_conv_int8(gp, to_device(x, layout), y, n, h, w, layout, W.SPLIT, ws)
    torch.cuda.synchronize()
    return from_device_nchw(y, layout)


@pytest.mark.parametrize("layout", [W.NHWC, W.NCHW])
@pytest.mark.parametrize("shape", SHAPES)
def test_streamk_bitexact_and_repeatable(shape, layout):
    torch = torch_dev()
    n, cin, cout, h, w = shape
    x, gp, op = _plans(shape, 31 + cin, relu=cout % 2 == 0)
    W.wino_f4_plan_set_tap_kernel(gp, W.TAP_ROWS_STREAMK)
    assert W.wino_f4_tap_kernel_choice(gp, n, h, w) == W.TAP_ROWS_STREAMK
    vq_bytes, total = _split_bytes(shape)
    assert W.wino_f4_workspace_bytes(gp, n, h, w) == total
    ref = tapwise.conv_int8(x, op)
    # poisoned workspace: the input transform must zero the counters itself
    ws = torch.full((total,), -1, dtype=torch.int8, device="cuda")
    for call in range(2):
        got = _conv(gp, x, layout, ws)
        assert (got == ref).all(), f"call {call}: {(got != ref).sum()} bytes differ"
    # the split steps on their own: one input transform, two tap GEMMs
    xd = to_device(x, layout)
    W.wino_f4_input_transform(gp, xd, n, h, w, layout, ws)
    for call in range(2):
        y = empty_out(n, cout, h, w, layout)
        W.wino_f4_tap_gemm(gp, ws, y, n, h, w, layout)
        torch.cuda.synchronize()
        got = from_device_nchw(y, layout)
        assert (got == ref).all(), f"tap GEMM {call}: {(got != ref).sum()} bytes differ"
    # a workspace that holds Vq only: the unsplit kernel, the same bytes
    small = torch.empty(vq_bytes, dtype=torch.int8, device="cuda")
    assert (_conv(gp, x, layout, small) == ref).all()


def test_streamk_choice_rules():
    ncu = _ncu()
    f = np.random.default_rng(3).normal(0, 0.05, (64, 64, 3, 3)).astype(np.float32)
    gp = W.wino_f4_plan(f, [4] * 36, bias=None, out_shift=10)
    # below one round of blocks: AUTO keeps the 64x32 tap-resident kernel,
    # ROWS never splits, ROWS_STREAMK splits
    assert W.wino_f4_tap_kernel_choice(gp, 1, 32, 32) == W.TAP_RESIDENT_64X32
    W.wino_f4_plan_set_tap_kernel(gp, W.TAP_ROWS)
    assert W.wino_f4_tap_kernel_choice(gp, 1, 32, 32) == W.TAP_ROWS
    W.wino_f4_plan_set_tap_kernel(gp, W.TAP_ROWS_STREAMK)
    assert W.wino_f4_tap_kernel_choice(gp, 1, 32, 32) == W.TAP_ROWS_STREAMK
    # 64 output channels x (tiles / 64) blocks, here one block per 32 x 32
    # image: AUTO never splits (measured slower); the forced split applies
    # only where a last round is partial
    for blocks in (ncu, ncu + ncu // 2, 2 * ncu):
        W.wino_f4_plan_set_tap_kernel(gp, W.TAP_AUTO)
        assert W.wino_f4_tap_kernel_choice(gp, blocks, 32, 32) == W.TAP_ROWS, blocks
        W.wino_f4_plan_set_tap_kernel(gp, W.TAP_ROWS_STREAMK)
        want = W.TAP_ROWS if blocks % ncu == 0 else W.TAP_ROWS_STREAMK
        assert W.wino_f4_tap_kernel_choice(gp, blocks, 32, 32) == want, blocks
    with pytest.raises(W.WinoError):
        W.wino_f4_plan_set_tap_kernel(gp, W.TAP_ROWS_STREAMK + 1)
