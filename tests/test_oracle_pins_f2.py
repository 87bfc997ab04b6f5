"""Pins of the oracle's F(2x2, 3x3) pipeline (the same tap-wise scheme with
the F2 matrices of Sec. II: 4x4 input tiles at stride 2, 16 taps, 2x2 output
tiles) against facts fixed by the paper and by mathematics (no GPU)."""
from fractions import Fraction as Fr

import numpy as np
import pytest

from oracle import direct, f4, quant, tapwise

F2 = tapwise.F2


@pytest.mark.parametrize("h,w", [(8, 8), (13, 6), (1, 1), (5, 3), (2, 9)])
def test_float_f2_equals_direct(h, w):
    """Winograd F2 in float64 is an exact algorithm up to rounding."""
    rng = np.random.default_rng(h * 17 + w)
    x = rng.normal(size=(2, 4, h, w))
    f = rng.normal(size=(3, 4, 3, 3))
    yw = tapwise.conv_winograd_f64(x, f, m=2)
    yd = direct.conv_f64(x, f)
    assert yw.shape == yd.shape
    assert np.abs(yw - yd).max() / np.abs(yd).max() <= 1e-12


def test_f2_spec_shapes():
    assert (F2.m, F2.n, F2.ntap, F2.den) == (2, 4, 16, 2)
    assert F2.Gint == [[2, 0, 0], [1, 1, 1], [1, -1, 1], [0, 0, 2]]
    assert tapwise.tile_grid(7, 8, 2) == (4, 4)


def test_f2_plan_uq_matches_rational_definition():
    """Uq and e_G from the integer-mantissa implementation equal a per-element
    evaluation of U = G f G^T with Fractions straight from the definition."""
    rng = np.random.default_rng(12)
    f = rng.normal(0, 0.2, (3, 2, 3, 3)).astype(np.float32)
    f[0, 0, 2, 0] = np.float32(3e-29)          # wide exponent spread
    f[1, 0] = 0.0
    plan = tapwise.make_plan(f, [0] * 16, m=2)
    g = f4.G2
    U = {}
    for co in range(3):
        for ci in range(2):
            fr = [[Fr(float(f[co, ci, r, c])) for c in range(3)] for r in range(3)]
            for a in range(4):
                for b in range(4):
                    U[co, ci, a, b] = sum(g[a][r] * fr[r][c] * g[b][c] for r in range(3) for c in range(3))
    for t in range(16):
        a, b = divmod(t, 4)
        mx = max(abs(U[co, ci, a, b]) for co in range(3) for ci in range(2))
        assert plan["e_g"][t] == quant.cexp(mx)
        for co in range(3):
            for ci in range(2):
                assert plan["uq"][t, ci, co] == quant.quantize_exact(U[co, ci, a, b], plan["e_g"][t])


@pytest.mark.parametrize("seed,n,cin,cout,h,w,relu", [
    (0, 1, 1, 1, 1, 1, False), (1, 1, 2, 3, 3, 5, True), (2, 2, 3, 2, 9, 4, False),
    (3, 1, 3, 1, 2, 7, True), (4, 1, 2, 2, 8, 8, False)])
def test_f2_pipeline_batched_equals_naive(seed, n, cin, cout, h, w, relu):
    rng = np.random.default_rng(seed)
    x = rng.integers(-128, 128, (n, cin, h, w)).astype(np.int8)
    f = rng.normal(0, 0.3, (cout, cin, 3, 3)).astype(np.float32)
    b = rng.integers(-300, 301, cout)
    eb = [int(v) for v in rng.integers(0, 5, 16)]
    for s in (0, 4, 9):
        plan = tapwise.make_plan(f, eb, bias=b, out_shift=s, relu=relu, m=2)
        assert (tapwise.conv_int8(x, plan) == tapwise.conv_int8_naive(x, plan)).all()


def test_f2_input_transform_bound():
    """Every row of the F2 B^T has two entries of magnitude 1, so |V| <= 4 |d|
    (512 for int8 inputs), reached by a checkerboard of -128 / 127."""
    d = np.zeros((1, 1, 1, 1, 4, 4), dtype=np.int64)
    sign = np.array([[1, -1, -1, 1], [-1, 1, 1, -1], [-1, 1, 1, -1], [1, -1, -1, 1]])
    d[..., :, :] = np.where(sign > 0, 127, -128)
    v = tapwise.input_transform(d, F2)
    assert np.abs(v).max() <= 512
    rng = np.random.default_rng(0)
    x = rng.integers(-128, 128, (2, 3, 9, 9))
    assert np.abs(tapwise.input_transform(tapwise.input_tiles(x, F2), F2)).max() <= 512


def _f2_lossless(seed, corner_only):
    rng = np.random.default_rng(seed)
    n, cin, cout, h, w = 2, 3, 4, 9, 7
    s = 4
    fint = np.zeros((cout, cin, 3, 3), dtype=np.int64)
    if corner_only:
        fint[:, :, 0, 0] = rng.integers(-1, 2, (cout, cin))
    else:
        fint[:] = rng.integers(-1, 2, (cout, cin, 3, 3))
    f = (4.0 * 2.0 ** -s * fint).astype(np.float32)     # U 2^s = Gint f_int Gint^T
    return rng, n, cin, cout, h, w, s, fint, f


def test_f2_lossless_equals_direct_uniform_scales():
    """Binary inputs (|V| <= 4, e_B = 0 exact) and weights f = 4 2^-s f_int
    (|U 2^s| <= 9, e_G = -s exact): Y 2^e_o = sum x f exactly."""
    rng, n, cin, cout, h, w, s, fint, f = _f2_lossless(5, corner_only=False)
    x = rng.integers(0, 2, (n, cin, h, w)).astype(np.int8)
    plan = tapwise.make_plan(f, [0] * 16, e_g=[-s] * 16, m=2)
    assert int(np.abs(plan["uq"]).max()) <= 9
    assert plan["e_o"] == -s and plan["sh"] == [0] * 16
    z = tapwise.prequant_output(x, plan)
    assert (z == 4 * direct.conv_int(x, fint)).all()


def _f2_unequal_case():
    """Corner weights give U 2^s = outer(Gint[:,0]) f_int with magnitudes in
    {0, 1, 2, 4}; per-tap e_G = -s + log2 |.| makes Uq = +-1 exactly.  Inputs
    in {0, 8} with e_B in {2, 3} are exact too, so the alignment shifts
    differ across taps while the result must still be exact."""
    rng, n, cin, cout, h, w, s, fint, f = _f2_lossless(6, corner_only=True)
    col = [row[0] for row in F2.Gint]                  # [2, 1, 1, 0]
    e_g = []
    for t in range(16):
        mm = abs(col[t // 4] * col[t % 4])
        e_g.append(-s + (mm.bit_length() - 1 if mm else 0))
    e_b = [int(v) for v in rng.integers(2, 4, 16)]
    x = (8 * rng.integers(0, 2, (n, cin, h, w))).astype(np.int8)
    return x, f, fint, e_g, e_b, s


def test_f2_lossless_equals_direct_unequal_shifts():
    x, f, fint, e_g, e_b, s = _f2_unequal_case()
    plan = tapwise.make_plan(f, e_b, e_g=e_g, m=2)
    assert len(set(plan["sh"])) > 2
    z = tapwise.prequant_output(x, plan)
    ref = 4 * direct.conv_int(x, fint)
    scale = plan["e_o"] + s
    lhs = z * (2 ** scale) if scale >= 0 else z
    rhs = ref if scale >= 0 else ref * (2 ** -scale)
    assert (lhs == rhs).all()


def test_f2_lossless_detects_dropped_alignment():
    """Planted mistake: with every alignment shift set to 0 the unequal-shift
    lossless case no longer equals direct convolution."""
    x, f, fint, e_g, e_b, s = _f2_unequal_case()
    plan = tapwise.make_plan(f, e_b, e_g=e_g, m=2)
    plan["sh"] = [0] * 16
    z = tapwise.prequant_output(x, plan)
    ref = 4 * direct.conv_int(x, fint)
    scale = plan["e_o"] + s
    assert not (z * 2 ** max(scale, 0) == ref * 2 ** max(-scale, 0)).all()


def test_f2_detects_transposed_tap_exponents():
    """Planted mistake: reading the input exponent of tap (a, b) as (b, a)
    breaks the exact case when the exponents are asymmetric."""
    x, f, fint, e_g, e_b, s = _f2_unequal_case()
    e_b = [3 if (t // 4) < (t % 4) else 2 for t in range(16)]
    good = tapwise.make_plan(f, e_b, e_g=e_g, m=2)
    bad = tapwise.make_plan(f, e_b, e_g=e_g, m=2)
    bad["e_b"] = [e_b[(t % 4) * 4 + t // 4] for t in range(16)]
    ref = 4 * direct.conv_int(x, fint)
    zg = tapwise.prequant_output(x, good)
    zb = tapwise.prequant_output(x, bad)
    sc = good["e_o"] + s
    assert (zg * 2 ** max(sc, 0) == ref * 2 ** max(-sc, 0)).all()
    assert not (zb * 2 ** max(sc, 0) == ref * 2 ** max(-sc, 0)).all()


@pytest.mark.parametrize("seed", [0, 1])
def test_f2_quantization_error_bound(seed):
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 128, (1, 5, 9, 10)).astype(np.int8)
    f = rng.normal(0, 0.15, (4, 5, 3, 3)).astype(np.float32)
    eb = tapwise.calibrate_input_exps(x, m=2)
    plan = tapwise.make_plan(f, eb, m=2)
    y = tapwise.prequant_output(x, plan).astype(np.float64) * 2.0 ** plan["e_o"]
    ref = direct.conv_f64(x, f.astype(np.float64))
    bound = tapwise.quantization_error_bound(x, f, plan, clamped_slack=True)
    err = np.abs(y - ref)
    assert (err <= bound * (1 + 1e-9) + 1e-9).all()
    assert np.sqrt((err ** 2).mean()) < 0.5 * np.sqrt((ref ** 2).mean())


def test_f2_calibration_minimal_and_safe():
    rng = np.random.default_rng(9)
    x = rng.integers(-128, 128, (2, 3, 10, 9)).astype(np.int8)
    amax = tapwise.input_tap_absmax(x, m=2)
    eb = tapwise.calibrate_input_exps(x, m=2)
    assert len(eb) == 16
    for t in range(16):
        assert amax[t] <= 128 * 2 ** eb[t]
        if eb[t] > 0:
            assert amax[t] > 128 * 2 ** (eb[t] - 1)
    f = rng.normal(0, 0.2, (4, 3, 3, 3)).astype(np.float32)
    plan = tapwise.make_plan(f, eb, bias=rng.integers(-64, 65, 4), m=2)
    s = tapwise.calibrate_out_shift(x, plan)
    z = tapwise.prequant_output(x, plan)
    assert np.abs(z).max() <= 128 * 2 ** s
    assert s == 0 or np.abs(z).max() > 128 * 2 ** (s - 1)


def test_f2_epilogue_bound_dominates_actual_values():
    rng = np.random.default_rng(10)
    x = rng.integers(-128, 128, (1, 6, 8, 8)).astype(np.int8)
    f = rng.normal(0, 0.3, (3, 6, 3, 3)).astype(np.float32)
    eb = [int(v) for v in rng.integers(0, 5, 16)]
    plan = tapwise.make_plan(f, eb, bias=rng.integers(-64, 65, 3), out_shift=6, m=2)
    z = tapwise.prequant_output(x, plan)
    assert np.abs(z).max() + 32 <= tapwise.epilogue_bound(plan)


def test_f2_and_f4_differ_but_both_approximate():
    """The two transforms are different quantized approximations of the same
    convolution: on random data they disagree somewhere, yet both are within
    their error bounds of direct convolution."""
    rng = np.random.default_rng(3)
    x = rng.integers(0, 128, (1, 4, 8, 8)).astype(np.int8)
    f = rng.normal(0, 0.2, (3, 4, 3, 3)).astype(np.float32)
    ref = direct.conv_f64(x, f.astype(np.float64))
    outs = []
    for m in (4, 2):
        plan = tapwise.make_plan(f, tapwise.calibrate_input_exps(x, m=m), m=m)
        y = tapwise.prequant_output(x, plan).astype(np.float64) * 2.0 ** plan["e_o"]
        bound = tapwise.quantization_error_bound(x, f, plan, clamped_slack=True)
        assert (np.abs(y - ref) <= bound * (1 + 1e-9) + 1e-9).all()
        outs.append(y)
    assert not np.array_equal(outs[0], outs[1])
