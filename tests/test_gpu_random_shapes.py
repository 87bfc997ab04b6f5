"""GPU parity on shapes hypothesis draws (derandomized, so every run checks
the same cases): batch, channel counts (partial 64-channel blocks, several
k-chunks), image sizes (ragged tiles, images smaller than a tile), layout,
transform (F4 / F2), variant (SPLIT / FUSED), tap-GEMM kernel, ReLU and
output shift.  Every output
byte must equal the oracle's."""
import numpy as np
import pytest

import paper_2209_12982_amd as W
import workloads
from oracle import tapwise

from gpu_util import run_conv

hyp = pytest.importorskip("hypothesis")
from hypothesis import given, settings, strategies as st  # noqa: E402

pytestmark = pytest.mark.gpu

KERNELS_F4 = [W.TAP_AUTO, W.TAP_ROWS, W.TAP_WAVES, W.TAP_RESIDENT_64X32, W.TAP_RESIDENT_32X32,
              W.TAP_RESIDENT_16X16]


@settings(max_examples=160, deadline=None, derandomize=True)
@given(n=st.integers(1, 3), cin=st.integers(1, 150), cout=st.integers(1, 140), h=st.integers(1, 37),
       w=st.integers(1, 37), layout=st.sampled_from([W.NCHW, W.NHWC]), m=st.sampled_from([4, 2]),
       variant=st.sampled_from([W.SPLIT, W.FUSED]), kernel=st.sampled_from(KERNELS_F4), relu=st.booleans(),
       out_shift=st.integers(0, 14), signed=st.booleans(), seed=st.integers(0, 2 ** 31 - 1))
def test_random_shape_bitexact(n, cin, cout, h, w, layout, m, variant, kernel, relu, out_shift, signed, seed):
    torch_ok = pytest.importorskip("torch").cuda.is_available()
    if not torch_ok:
        pytest.skip("no GPU")
    x, f, b = workloads.random_case(seed % 1000, n, cin, cout, h, w, signed=signed, zero_frac=0.5)
    eb = tapwise.calibrate_input_exps(x, m=m)
    make = W.wino_f4_plan if m == 4 else W.wino_f2_plan
    gp = make(f, eb, bias=b, out_shift=out_shift, relu=relu)
    op = tapwise.make_plan(f, eb, bias=b, out_shift=out_shift, relu=relu, m=m)
    if m == 4:
        W.wino_f4_plan_set_tap_kernel(gp, kernel)
    y = run_conv(gp, x, layout, variant)
    ref = tapwise.conv_int8(x, op)
    assert (y == ref).all(), f"{(y != ref).sum()} mismatches"
