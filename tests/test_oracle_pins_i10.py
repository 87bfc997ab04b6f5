"""Pins of the oracle's int8/10 variant (Sec. V: int8 in the spatial domain,
10-bit integers in the Winograd domain) against facts fixed by the
definition and by mathematics.  Each names what it pins and which plausible
slip (a clamp or scale left at 8 bits, a wrong range) would fail it."""
from fractions import Fraction as Fr

import numpy as np
import pytest

from oracle import direct, f4, quant, tapwise


def test_quantizer_range_and_scale_rule():
    """n = 10 in Eq. quant: [-512, 511], s = x_max / 2^9, power-of-two rule."""
    assert quant.qrange(10) == (-512, 511) and quant.qrange(8) == (-128, 127)
    assert quant.quantize_exact(Fr(1023, 2), 0, bits=10) == 511      # R(511.5) = 512 -> 511
    assert quant.quantize_exact(-512, 0, bits=10) == -512
    assert quant.quantize_exact(Fr(-1025, 2), 0, bits=10) == -512    # R(-512.5) = -512
    assert quant.quantize_exact(1023, 1, bits=10) == 511
    assert quant.quantize_exact(300, 0, bits=10) == 300               # would clamp at 8 bits
    assert quant.quantize_exact(300, 0) == 127
    assert quant.cexp(512, 10) == 0 and quant.cexp(Fr(512) + Fr(1, 10 ** 20), 10) == 1
    assert quant.cexp(1, 10) == -9 and quant.cexp(256, 10) == -1
    for a in [Fr(3, 7), Fr(1000), Fr(12768), Fr(1, 3)]:
        e = quant.cexp(a, 10)
        assert a <= 512 * Fr(2) ** e and a > 512 * Fr(2) ** (e - 1)
        assert e == quant.cexp(a) - 2                                 # 2^9 = 4 * 2^7


def test_plan_uq_10bit_matches_rational_definition():
    """Uq and e_G of a 10-bit plan equal a per-element evaluation with
    Fractions of U = G f G^T from the printed G."""
    rng = np.random.default_rng(12)
    f = rng.normal(0, 0.2, (3, 2, 3, 3)).astype(np.float32)
    f[0, 0, 1, 1] = np.float32(1e-30)
    plan = tapwise.make_plan(f, [0] * 36, bits=10)
    g = f4.G4
    U = {}
    for co in range(3):
        for ci in range(2):
            fr = [[Fr(float(f[co, ci, r, c])) for c in range(3)] for r in range(3)]
            for a in range(6):
                for b in range(6):
                    U[co, ci, a, b] = sum(g[a][r] * fr[r][c] * g[b][c] for r in range(3) for c in range(3))
    for t in range(36):
        a, b = divmod(t, 6)
        mx = max(abs(U[co, ci, a, b]) for co in range(3) for ci in range(2))
        assert plan["e_g"][t] == quant.cexp(mx, 10)
        for co in range(3):
            for ci in range(2):
                assert plan["uq"][t, ci, co] == quant.quantize_exact(U[co, ci, a, b], plan["e_g"][t], bits=10)
    assert int(np.abs(plan["uq"]).max()) > 127                        # uses the wider range


@pytest.mark.parametrize("m", [4, 2])
@pytest.mark.parametrize("seed,n,cin,cout,h,w,relu", [
    (0, 1, 1, 1, 1, 1, False), (1, 1, 2, 3, 3, 5, True), (2, 2, 3, 2, 9, 4, False), (3, 1, 3, 1, 2, 7, True)])
def test_pipeline_10bit_batched_equals_naive(m, seed, n, cin, cout, h, w, relu):
    rng = np.random.default_rng(seed)
    ntap = (m + 2) ** 2
    x = rng.integers(-128, 128, (n, cin, h, w)).astype(np.int8)
    f = rng.normal(0, 0.3, (cout, cin, 3, 3)).astype(np.float32)
    b = rng.integers(-3000, 3001, cout)
    eb = [int(v) for v in rng.integers(0, 7, ntap)]
    for s in (0, 7, 14):
        plan = tapwise.make_plan(f, eb, bias=b, out_shift=s, relu=relu, m=m, bits=10)
        assert (tapwise.conv_int8(x, plan) == tapwise.conv_int8_naive(x, plan)).all()


def _lossless_case(seed):
    """Inputs in [-4, 4] (|V| <= 10 * 10 * 4 = 400 for F4) and centre-only
    weights f = 576 2^-s k with k in [-31, 31] (U 2^s = k G24[:,1] G24[:,1]^T,
    |.| <= 16 * 31 = 496): every Winograd-domain value fits 10 bits."""
    rng = np.random.default_rng(seed)
    n, cin, cout, h, w, s = 2, 3, 4, 10, 7, 5
    k = np.zeros((cout, cin, 3, 3), dtype=np.int64)
    k[:, :, 1, 1] = rng.integers(-31, 32, (cout, cin))
    k[0, 0, 1, 1] = 31
    f = (576.0 * 2.0 ** -s * k).astype(np.float32)
    x = rng.integers(-4, 5, (n, cin, h, w)).astype(np.int8)
    return x, f, k, s


def test_lossless_10bit_equals_direct():
    """With e_B = 0 and e_G = -s every quantization is exact at 10 bits, so
    Y 2^e_o equals direct convolution; the calibrated 10-bit scales find
    such a plan by themselves.  At 8 bits the same case clamps (|V| up to
    400, |U 2^s| up to 496), which the comparison must detect."""
    x, f, k, s = _lossless_case(1)
    ref = 576 * direct.conv_int(x, k)                       # = 2^s * sum x f
    v = tapwise.input_tap_absmax(x)
    assert max(v) > 127 and max(v) <= 400
    plan = tapwise.make_plan(f, [0] * 36, e_g=[-s] * 36, bits=10)
    assert plan["e_o"] == -s
    assert (tapwise.prequant_output(x, plan) == ref).all()
    # calibrated 10-bit exponents: still exact
    eb = tapwise.calibrate_input_exps(x, bits=10)
    assert eb == [0] * 36
    cal = tapwise.make_plan(f, eb, bits=10)
    z = tapwise.prequant_output(x, cal)
    sc = cal["e_o"] + s
    assert (z * 2 ** max(sc, 0) == ref * 2 ** max(-sc, 0)).all()
    # the same tables at 8 bits are not lossless
    p8 = tapwise.make_plan(f, [0] * 36, e_g=[-s] * 36)
    assert not (tapwise.prequant_output(x, p8) == ref).all()


def test_lossless_10bit_f2():
    """F2: Bt rows have |.|-sums <= 2, so inputs in [-128, 127] give
    |V| <= 512 -- all but +512 fit [-512, 511]; with inputs in [-127, 127]
    and centre-only weights f = 4 2^-s k (|U 2^s| <= |k| <= 127) the
    10-bit F2 pipeline is exact."""
    rng = np.random.default_rng(3)
    n, cin, cout, h, w, s = 1, 2, 3, 7, 9, 3
    k = np.zeros((cout, cin, 3, 3), dtype=np.int64)
    k[:, :, 1, 1] = rng.integers(-127, 128, (cout, cin))
    f = (4.0 * 2.0 ** -s * k).astype(np.float32)
    x = rng.integers(-127, 128, (n, cin, h, w)).astype(np.int8)
    plan = tapwise.make_plan(f, [0] * 16, e_g=[-s] * 16, m=2, bits=10)
    assert (tapwise.prequant_output(x, plan) == 4 * direct.conv_int(x, k)).all()
    p8 = tapwise.make_plan(f, [0] * 16, e_g=[-s] * 16, m=2)
    assert not (tapwise.prequant_output(x, p8) == 4 * direct.conv_int(x, k)).all()


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_quantization_error_bound_10bit(seed):
    """The analytic per-output bound of the two tap quantizations holds at 10
    bits, and the error is well below the 8-bit error (two more bits per
    operand: about 4x smaller)."""
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 128, (1, 6, 9, 11)).astype(np.int8)
    f = rng.normal(0, 0.15, (5, 6, 3, 3)).astype(np.float32)
    ref = direct.conv_f64(x, f.astype(np.float64))
    errs = {}
    for bits in (8, 10):
        eb = tapwise.calibrate_input_exps(x, bits=bits)
        plan = tapwise.make_plan(f, eb, bits=bits)
        y = tapwise.prequant_output(x, plan).astype(np.float64) * 2.0 ** plan["e_o"]
        bound = tapwise.quantization_error_bound(x, f, plan, clamped_slack=True)
        err = np.abs(y - ref)
        assert (err <= bound * (1 + 1e-9) + 1e-9).all()
        errs[bits] = np.sqrt((err ** 2).mean())
    assert errs[10] < 0.4 * errs[8]


def test_calibration_10bit_minimal_and_safe():
    rng = np.random.default_rng(4)
    x = rng.integers(-128, 128, (2, 3, 10, 9)).astype(np.int8)
    amax = tapwise.input_tap_absmax(x)
    eb = tapwise.calibrate_input_exps(x, bits=10)
    for t in range(36):
        assert amax[t] <= 512 * 2 ** eb[t]
        if eb[t] > 0:
            assert amax[t] > 512 * 2 ** (eb[t] - 1)
    assert eb == [max(0, e - 2) for e in tapwise.calibrate_input_exps(x)]


def test_epilogue_bound_10bit_dominates():
    """The bound uses the 10-bit operand range: it dominates |Y + bias| on
    inputs that drive Vq to the 10-bit rails."""
    rng = np.random.default_rng(8)
    x = rng.choice(np.array([-128, 127], np.int8), (1, 8, 8, 8))
    f = rng.normal(0, 0.3, (3, 8, 3, 3)).astype(np.float32)
    plan = tapwise.make_plan(f, [0] * 36, bias=rng.integers(-64, 65, 3), out_shift=6, bits=10)
    z = tapwise.prequant_output(x, plan)
    v = tapwise.input_taps_quantized(x, plan["e_b"], bits=10)
    assert np.abs(v).max() == 512                                      # rails reached
    assert np.abs(z).max() + 32 <= tapwise.epilogue_bound(plan)
