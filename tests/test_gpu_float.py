"""The unquantized fp32 Winograd F(4x4,3x3) stage (wino_f4_conv_float)
against the oracle's float64 Winograd F4 and its direct convolution: every
intermediate of that stage is an fp32 value, held to a normwise relative
error max|y - ref| / max|ref| <= 1e-5.

Tolerance: each fp32 operation rounds by at most 2^-24 (6e-8) relative; the
transforms take at most 6 + 6 terms per pass with coefficients up to 5 (B^T)
and 8 (A^T), and M sums 16-channel blocks.  A float32 evaluation of the same
algorithm on the CPU (numpy) stays at 1.8e-6 (C1, 16 channels) and 4.4e-6
(C2, 64 channels) against float64, under the 1e-5 bound."""
import numpy as np
import pytest

import paper_2209_12982_amd as W
import workloads
from oracle import direct, tapwise

from gpu_util import from_device_nchw, to_device, torch_dev

pytestmark = pytest.mark.gpu

TOL = 1e-5


def _run(x, f, layout):
    torch = torch_dev()
    n, cin, h, w = x.shape
    cout = f.shape[0]
    xd = to_device(x, layout)
    wd = torch.from_numpy(np.ascontiguousarray(f, dtype=np.float32)).cuda()
    shape = (n, cout, h, w) if layout == W.NCHW else (n, h, w, cout)
    y = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
    W.wino_f4_conv_float(xd, wd, y, n, cin, cout, h, w, layout)
    torch.cuda.synchronize()
    return from_device_nchw(y, layout).astype(np.float64)


def _rel(y, ref):
    return np.abs(y - ref).max() / np.abs(ref).max()


@pytest.mark.parametrize("layout", [W.NCHW, W.NHWC])
@pytest.mark.parametrize("case", ["C1", "C2_one_image", "ragged"])
def test_float_winograd_within_1e5(case, layout):
    if case == "ragged":
        rng = np.random.default_rng(7)
        x = workloads.draw_activations(rng, (2, 24, 13, 22), "halfnormal24", 0.5)
        f = rng.normal(0, np.sqrt(2 / (9 * 24)), (40, 24, 3, 3)).astype(np.float32)
    else:
        x, layers = workloads.generate(case.split("_")[0])
        f = layers[0][0]
        if case == "C2_one_image":
            x = x[:1]
    y = _run(x, f, layout)
    assert np.isfinite(y).all(), "some output was not written"
    ref = tapwise.conv_winograd_f64(x, f)
    assert _rel(y, ref) <= TOL
    # the float Winograd algorithm is exact convolution up to rounding
    assert _rel(y, direct.conv_f64(x, f)) <= TOL


def test_float_winograd_small_images():
    # H, W not multiples of 4 and smaller than a tile: outputs outside the
    # image are dropped, the zero padding enters the transform
    rng = np.random.default_rng(11)
    for h, w in [(1, 1), (2, 3), (5, 5), (3, 9)]:
        x = rng.integers(-128, 128, (1, 3, h, w)).astype(np.int8)
        f = rng.normal(0, 0.3, (5, 3, 3, 3)).astype(np.float32)
        for layout in (W.NCHW, W.NHWC):
            y = _run(x, f, layout)
            assert _rel(y, direct.conv_f64(x, f)) <= TOL, (h, w, layout)


def test_float_winograd_argument_errors():
    torch = torch_dev()
    x = torch.zeros(64, dtype=torch.int8, device="cuda")
    wd = torch.zeros(9 * 4, dtype=torch.float32, device="cuda")
    y = torch.full((64,), 5.0, dtype=torch.float32, device="cuda")
    with pytest.raises(W.WinoError):
        W.wino_f4_conv_float(x, wd, y, 1, 0, 4, 4, 4, W.NCHW)          # cin < 1
    with pytest.raises(W.WinoError):
        W.wino_f4_conv_float(x, wd, y, 1, 1, 4, 4, 4, 7)               # bad layout
    W.wino_f4_conv_float(x, wd, y, 0, 1, 4, 4, 4, W.NCHW)              # empty batch: nothing written
    torch.cuda.synchronize()
    assert (y.cpu().numpy() == 5.0).all()
