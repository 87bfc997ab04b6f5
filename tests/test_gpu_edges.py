"""Edge cases of the online path through the C ABI: empty batches and
images (nothing is written), the size limits and a short workspace (refused
before any launch, with the documented status), and a layer with many input
channels against the oracle."""
import numpy as np
import pytest

import paper_2209_12982_amd as W
import workloads
from oracle import tapwise

from gpu_util import run_conv, torch_dev, workspace

pytestmark = pytest.mark.gpu

PLANS = [("f4", W.wino_f4_plan, 36), ("f2", W.wino_f2_plan, 16), ("f4_i10", W.wino_f4_plan_i10, 36),
         ("f2_i10", W.wino_f2_plan_i10, 16)]


@pytest.mark.parametrize("name,make,ntap", PLANS)
@pytest.mark.parametrize("layout", [W.NCHW, W.NHWC])
@pytest.mark.parametrize("n,h,w", [(0, 8, 8), (1, 0, 8), (2, 8, 0)])
def test_empty_input_writes_nothing(name, make, ntap, layout, n, h, w):
    torch = torch_dev()
    f = np.random.default_rng(1).normal(0, 0.2, (8, 4, 3, 3)).astype(np.float32)
    plan = make(f, [0] * ntap)
    assert W.wino_f4_workspace_bytes(plan, n, h, w) == 0
    x = torch.zeros(16, dtype=torch.int8, device="cuda")           # never read
    y = torch.full((64,), 77, dtype=torch.int8, device="cuda")     # never written
    W.wino_f4_conv_int8(plan, x, y, n, h, w, layout, W.SPLIT, None)
    W.wino_f4_input_transform(plan, x, n, h, w, layout, None)
    torch.cuda.synchronize()
    assert (y.cpu().numpy() == 77).all()


def test_limits_and_workspace_are_refused():
    """The C ABI's own checks, called directly with buffers far smaller than
    the sizes (nothing may be launched)."""
    import ctypes
    torch = torch_dev()
    f = np.zeros((4, 4, 3, 3), np.float32)
    plan = W.wino_f4_plan(f, [0] * 36)
    x = torch.zeros(16, dtype=torch.int8, device="cuda")
    y = torch.zeros(16, dtype=torch.int8, device="cuda")
    ws = torch.zeros(16, dtype=torch.int8, device="cuda")
    lib = W.load_library()
    P = ctypes.c_void_p
    st = torch.cuda.current_stream().cuda_stream
    cases = [
        ((1, 65537, 8), -2),          # image side beyond 65536
        ((1, 32768, 32768), -2),      # 2^26 tiles
        ((-1, 8, 8), -1),             # negative size
        ((1, 64, 64), -5),            # workspace of 16 bytes
    ]
    for (n, h, w), status in cases:
        got = lib.wino_f4_conv_int8(plan.handle, P(x.data_ptr()), P(y.data_ptr()), n, h, w, W.NHWC, W.SPLIT,
                                    P(ws.data_ptr()), 16, P(st))
        assert got == status, (n, h, w)
    assert lib.wino_f4_conv_int8(plan.handle, P(x.data_ptr()), P(y.data_ptr()), 1, 8, 8, 7, W.SPLIT,
                                 P(ws.data_ptr()), 16, P(st)) == -1               # unknown layout
    torch.cuda.synchronize()
    assert (y.cpu().numpy() == 0).all()


def test_binding_refuses_buffers_a_kernel_cannot_use():
    """Host tensors, wrong dtypes, non-contiguous views and buffers shorter
    than the call's sizes are refused by the binding before the C ABI sees
    a pointer."""
    torch = torch_dev()
    f = np.zeros((4, 4, 3, 3), np.float32)
    plan = W.wino_f4_plan(f, [0] * 36)
    n, h, w = 1, 8, 8
    x = torch.zeros((n, 4, h, w), dtype=torch.int8, device="cuda")
    y = torch.full((n, 4, h, w), 7, dtype=torch.int8, device="cuda")
    ws = torch.empty(W.wino_f4_workspace_bytes(plan, n, h, w), dtype=torch.int8, device="cuda")
    bad_inputs = [
        x.cpu(),                                          # host memory
        x.to(torch.int32),                                # wrong dtype
        torch.zeros((n, 4, h, 2 * w), dtype=torch.int8, device="cuda")[..., ::2],   # strided view
        torch.zeros(16, dtype=torch.int8, device="cuda"),  # too short
    ]
    for bad in bad_inputs:
        with pytest.raises(ValueError):
            W.wino_f4_conv_int8(plan, bad, y, n, h, w, W.NCHW, W.SPLIT, ws)
        with pytest.raises(ValueError):
            W.wino_f4_conv_int8(plan, x, bad, n, h, w, W.NCHW, W.SPLIT, ws)
    with pytest.raises(ValueError):
        W.direct_conv_int8(x, torch.zeros(8, dtype=torch.int8, device="cuda"), None, y, n, 4, 4, h, w)
    torch.cuda.synchronize()
    assert (y.cpu().numpy() == 7).all()


@pytest.mark.parametrize("make,m", [(W.wino_f4_plan, 4), (W.wino_f2_plan, 2), (W.wino_f4_plan_i10, 4)])
def test_deep_channels_bitexact(make, m):
    """2048 input channels (32 k-chunks) and 96 output channels on a ragged
    9 x 7 image: long accumulations and padded output channels, SPLIT and
    (8-bit plans) FUSED."""
    n, cin, cout, h, w = 1, 2048, 96, 9, 7
    x, f, b = workloads.random_case(71, n, cin, cout, h, w, signed=True)
    bits = 10 if make is W.wino_f4_plan_i10 else 8
    eb = tapwise.calibrate_input_exps(x, m=m, bits=bits)
    plan = make(f, eb, bias=b, out_shift=11)
    ref = tapwise.conv_int8(x, tapwise.make_plan(f, eb, bias=b, out_shift=11, m=m, bits=bits))
    for layout in (W.NCHW, W.NHWC):
        assert (run_conv(plan, x, layout) == ref).all()
        if bits == 8:
            assert (run_conv(plan, x, layout, W.FUSED) == ref).all()


@pytest.mark.parametrize("shape,macs", [(16, 8 * 16 * 16 * 64), (32, 4 * 32 * 32 * 32)])
def test_mfma_probe_counts_its_operations(shape, macs):
    """The matrix-core probe the bench times reports 2 operations per
    multiply-add of its launch and never writes its sink."""
    torch = torch_dev()
    sink = torch.full((4,), 5, dtype=torch.int32, device="cuda")
    ops = W.wino_probe_mfma_int8(shape, 3, 2, sink)
    torch.cuda.synchronize()
    assert ops == 2 * macs * 4 * 2 * 3
    assert (sink.cpu().numpy() == 5).all()
