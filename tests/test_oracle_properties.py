"""Property tests of the oracle over random shapes and data (CPU).

The fixed-seed pins in test_oracle_pins.py check each property on a few
hand-picked cases; here hypothesis draws the shapes, the data and the tap
exponents, so that a mistake that only shows for some geometry (a tile
count, a border, a channel count) is found too:

* the float64 Winograd F(4x4,3x3) equals direct convolution (Sec. II);
* the tap-major integer pipeline equals its per-tile scalar formulation;
* with lossless quantization (binary inputs, weights 576 2^-s f_int on the
  2x2 corner, e_B = 0, e_G = -s) the integer pipeline equals direct
  convolution exactly (Sec. III scheme with no rounding);
* the analytic per-output error bound holds for any data without clamping.
"""
import numpy as np
import pytest

hyp = pytest.importorskip("hypothesis")
from hypothesis import given, settings, strategies as st  # noqa: E402

from oracle import direct, tapwise  # noqa: E402

SHAPES = st.tuples(st.integers(1, 2), st.integers(1, 4), st.integers(1, 4), st.integers(1, 11),
                   st.integers(1, 11))
SEEDS = st.integers(0, 2 ** 31 - 1)


@settings(max_examples=25, deadline=None)
@given(shape=SHAPES, seed=SEEDS)
def test_float_winograd_equals_direct(shape, seed):
    n, cin, cout, h, w = shape
    rng = np.random.default_rng(seed)
    x = rng.integers(-128, 128, (n, cin, h, w)).astype(np.int8)
    f = rng.normal(0, 0.5, (cout, cin, 3, 3)).astype(np.float32)
    ref = direct.conv_f64(x, f)
    got = tapwise.conv_winograd_f64(x, f)
    assert np.abs(got - ref).max() <= 1e-9 * max(1.0, np.abs(ref).max())


@settings(max_examples=25, deadline=None)
@given(shape=SHAPES, seed=SEEDS, relu=st.booleans(), out_shift=st.integers(0, 14))
def test_batched_pipeline_equals_per_tile_loops(shape, seed, relu, out_shift):
    n, cin, cout, h, w = shape
    rng = np.random.default_rng(seed)
    x = rng.integers(-128, 128, (n, cin, h, w)).astype(np.int8)
    f = rng.normal(0, 0.3, (cout, cin, 3, 3)).astype(np.float32)
    b = rng.integers(-300, 301, cout)
    eb = [int(v) for v in rng.integers(0, 9, 36)]
    plan = tapwise.make_plan(f, eb, bias=b, out_shift=out_shift, relu=relu)
    assert (tapwise.conv_int8(x, plan) == tapwise.conv_int8_naive(x, plan)).all()


@settings(max_examples=25, deadline=None)
@given(shape=SHAPES, seed=SEEDS, s=st.integers(0, 8))
def test_lossless_case_equals_direct(shape, seed, s):
    n, cin, cout, h, w = shape
    rng = np.random.default_rng(seed)
    fint = np.zeros((cout, cin, 3, 3), dtype=np.int64)
    fint[:, :, :2, :2] = rng.integers(-1, 2, (cout, cin, 2, 2))
    f = (576.0 * 2.0 ** -s * fint).astype(np.float32)
    x = rng.integers(0, 2, (n, cin, h, w)).astype(np.int8)
    plan = tapwise.make_plan(f, [0] * 36, e_g=[-s] * 36)
    z = tapwise.prequant_output(x, plan)
    assert plan["e_o"] == -s
    assert (z == 576 * direct.conv_int(x, fint)).all()


@settings(max_examples=15, deadline=None)
@given(shape=SHAPES, seed=SEEDS)
def test_error_bound_holds(shape, seed):
    n, cin, cout, h, w = shape
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 40, (n, cin, h, w)).astype(np.int8)
    f = rng.normal(0, 0.2, (cout, cin, 3, 3)).astype(np.float32)
    eb = tapwise.calibrate_input_exps(x)
    plan = tapwise.make_plan(f, eb)
    real = tapwise.prequant_output(x, plan).astype(np.float64) * 2.0 ** plan["e_o"]
    bound = tapwise.quantization_error_bound(x, f, plan, clamped_slack=True)
    assert (np.abs(real - direct.conv_f64(x, f)) <= bound + 1e-9).all()
