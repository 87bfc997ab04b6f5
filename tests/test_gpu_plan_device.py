"""GPU parity of the plans whose weight transform runs on the device
(wino_f4_plan_device / wino_f2_plan_device from fp32 weights, and
wino_f4_plan_int8 / wino_f2_plan_int8 from int8 spatial weights f_hat =
w * 2^e_f) against the oracle's exact plan, table for table and bit for bit,
and convolutions through them against the oracle's integer pipeline."""
import numpy as np
import pytest

import paper_2209_12982_amd as W
import workloads
from oracle import direct, tapwise

from gpu_util import run_conv, torch_dev

pytestmark = pytest.mark.gpu

MS = [4, 2]
SHAPES = [(1, 1), (3, 5), (70, 33), (64, 64), (130, 200), (256, 256)]   # (cin, cout)


def _ntap(m):
    return (m + 2) ** 2


def _expected(f, eb, m, e_g=None, bias=None, out_shift=0):
    o = tapwise.make_plan(f, eb, e_g=e_g, bias=bias, out_shift=out_shift, m=m)
    bits = 32 if tapwise.epilogue_bound(o) < 2 ** 31 and out_shift <= 31 else 64
    return o, bits


def _check_tables(plan, o, bits):
    info = W.wino_f4_plan_info(plan, with_uq=True)
    assert info["e_g"] == o["e_g"]
    assert info["sh"] == o["sh"]
    assert info["e_o"] == o["e_o"]
    assert info["epilogue_bits"] == bits
    assert (info["uq"] == o["uq"]).all(), f"{(info['uq'] != o['uq']).sum()} Uq mismatches"


def _device_plan(f, eb, m, **kw):
    torch = torch_dev()
    wd = torch.from_numpy(np.ascontiguousarray(f, dtype=np.float32)).cuda()
    fn = W.wino_f4_plan_device if m == 4 else W.wino_f2_plan_device
    return fn(wd, eb, **kw)


def _int8_plan(wi, e_f, eb, m, **kw):
    torch = torch_dev()
    wd = torch.from_numpy(np.ascontiguousarray(wi, dtype=np.int8)).cuda()
    fn = W.wino_f4_plan_int8 if m == 4 else W.wino_f2_plan_int8
    return fn(wd, e_f, eb, **kw)


def _eb(m, seed):
    return [int(v) for v in np.random.default_rng(seed).integers(0, 5, _ntap(m))]


@pytest.mark.parametrize("m", MS)
@pytest.mark.parametrize("shape", SHAPES)
def test_device_plan_tables_match_oracle(m, shape):
    cin, cout = shape
    rng = np.random.default_rng(cin * 1000 + cout)
    f = (rng.standard_normal((cout, cin, 3, 3)) * np.sqrt(2.0 / (9 * cin))).astype(np.float32)
    eb = _eb(m, 3)
    print(f"device plan F{m} cin={cin} cout={cout}", flush=True)
    plan = _device_plan(f, eb, m)
    _check_tables(plan, *_expected(f, eb, m))


def _adversarial(seed, cin, cout):
    """Dyadic weights (many exact rounding ties), taps whose maximum sits
    exactly on a power-of-two bound or one ulp above it, and mixed scales."""
    rng = np.random.default_rng(seed)
    kind = rng.integers(0, 5, (cout, cin, 3, 3))
    ud = rng.integers(-128, 129, (cout, cin, 3, 3)).astype(np.float32)
    ud2 = rng.integers(-128, 129, (cout, cin, 3, 3)).astype(np.float32)
    sgn = np.where(rng.integers(0, 2, (cout, cin, 3, 3)) == 0, -1.0, 1.0).astype(np.float32)
    f = np.zeros((cout, cin, 3, 3), np.float32)
    f = np.where(kind == 1, np.ldexp(ud, -5), f)
    f = np.where(kind == 2, sgn * np.float32(0.25) * (np.float32(1) + np.ldexp(np.float32(1), -23) * (np.abs(ud) % 3)), f)
    f = np.where(kind == 3, sgn * np.float32(16.0), f)
    f = np.where(kind == 4, np.ldexp(ud, -12) + np.ldexp(ud2, -40), f)
    return f.astype(np.float32)


@pytest.mark.parametrize("m", MS)
@pytest.mark.parametrize("seed", range(6))
def test_device_plan_adversarial_weights(m, seed):
    cin, cout = [(1, 1), (2, 3), (9, 7), (64, 5), (5, 70), (33, 33)][seed]
    f = _adversarial(100 + seed, cin, cout)
    eb = _eb(m, seed)
    plan = _device_plan(f, eb, m)
    _check_tables(plan, *_expected(f, eb, m))


@pytest.mark.parametrize("m", MS)
def test_device_plan_cancellation(m):
    """Terms of 1e6 that cancel around tiny ones: the double approximation of
    a sum is then far from every term, and only the exact expansion decides."""
    rng = np.random.default_rng(7)
    cout, cin = 5, 4
    f = np.zeros((cout, cin, 3, 3), np.float32)
    f[:, :, 0, 0], f[:, :, 0, 2] = 1e6, -1e6
    f[:, :, 0, 1] = rng.uniform(-1, 1, (cout, cin)) * 1e-6
    f[:, :, 1, 1] = rng.uniform(-1, 1, (cout, cin))
    f[:, :, 2, 0], f[:, :, 2, 2] = 3e6, -3e6
    f[:, :, 1, 0], f[:, :, 1, 2] = -1e6, 1e6
    eb = [0] * _ntap(m)
    o = tapwise.make_plan(f, eb, m=m)
    if tapwise.epilogue_bound(o) >= 2 ** 62:
        # the tap exponents spread too far for any integer epilogue: both refuse
        with pytest.raises(W.WinoError) as e:
            _device_plan(f, eb, m)
        assert e.value.status == -3
        # the weight tables themselves still agree, with the taps' exponents given
        plan = _device_plan(f, eb, m, w_exp=[min(max(v, -20), 20) for v in o["e_g"]])
        o2, bits2 = _expected(f, eb, m, e_g=[min(max(v, -20), 20) for v in o["e_g"]])
        _check_tables(plan, o2, bits2)
    else:
        _check_tables(_device_plan(f, eb, m), o, 32 if tapwise.epilogue_bound(o) < 2 ** 31 else 64)


@pytest.mark.parametrize("m", MS)
def test_device_plan_given_tap_exponents(m):
    rng = np.random.default_rng(11)
    f = (rng.standard_normal((40, 24, 3, 3)) * 0.1).astype(np.float32)
    eg = [int(v) for v in rng.integers(-12, -4, _ntap(m))]
    eb = _eb(m, 12)
    b = rng.integers(-500, 500, 40)
    plan = _device_plan(f, eb, m, w_exp=eg, bias=b, out_shift=9)
    _check_tables(plan, *_expected(f, eb, m, e_g=eg, bias=b, out_shift=9))


@pytest.mark.parametrize("m", MS)
@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5"])
def test_device_plan_config_weights(m, name):
    x, layers = workloads.generate(name)
    for k, (f, b, spec) in enumerate(layers):
        eb = _eb(m, k)
        print(f"{name} layer {k} F{m}", flush=True)
        plan = _device_plan(f, eb, m, bias=b)
        _check_tables(plan, *_expected(f, eb, m, bias=b))


@pytest.mark.parametrize("m", MS)
@pytest.mark.parametrize("layout", [W.NCHW, W.NHWC])
def test_conv_through_device_plan(m, layout):
    n, cin, cout, h, w = 2, 70, 80, 13, 18
    x, f, b = workloads.random_case(31, n, cin, cout, h, w, signed=True)
    eb = tapwise.calibrate_input_exps(x, m=m)
    plan = _device_plan(f, eb, m, bias=b, out_shift=8, relu=True)
    o = tapwise.make_plan(f, eb, bias=b, out_shift=8, relu=True, m=m)
    y = run_conv(plan, x, layout)
    assert (y == tapwise.conv_int8(x, o)).all()


def test_device_plan_rejects_non_finite():
    torch = torch_dev()
    for bad in (np.nan, np.inf, -np.inf):
        f = np.zeros((3, 2, 3, 3), np.float32)
        f[1, 1, 2, 0] = bad
        for fn in (W.wino_f4_plan_device, W.wino_f2_plan_device):
            ntap = 36 if fn is W.wino_f4_plan_device else 16
            with pytest.raises(W.WinoError) as e:
                fn(torch.from_numpy(f).cuda(), [0] * ntap)
            assert e.value.status == -1


# ---------------------------------------------------------------- int8 f_hat

def _int8_weights(seed, cout, cin):
    rng = np.random.default_rng(seed)
    wi = rng.integers(-128, 128, (cout, cin, 3, 3)).astype(np.int8)
    wi.flat[0] = -128
    wi.flat[-1] = 127
    return wi


def _f_hat(wi, e_f):
    return np.ldexp(wi.astype(np.float32), e_f).astype(np.float32)


@pytest.mark.parametrize("m", MS)
@pytest.mark.parametrize("e_f", [-100, -20, -7, 0, 5, 100])
@pytest.mark.parametrize("shape", [(1, 1), (13, 6), (64, 64), (130, 70)])
def test_int8_plan_tables_match_oracle(m, e_f, shape):
    cin, cout = shape
    wi = _int8_weights(cin + cout + e_f + 200, cout, cin)
    eb = _eb(m, 5)
    plan = _int8_plan(wi, e_f, eb, m)
    _check_tables(plan, *_expected(_f_hat(wi, e_f), eb, m))


@pytest.mark.parametrize("m", MS)
def test_int8_plan_sparse_and_zero_taps(m):
    """All-zero weights (every tap exponent 0), and one non-zero weight per
    kernel position so that some taps are all zero."""
    eb = _eb(m, 6)
    wi = np.zeros((5, 4, 3, 3), np.int8)
    _check_tables(_int8_plan(wi, -7, eb, m), *_expected(_f_hat(wi, -7), eb, m))
    wi[:, :, 0, 0] = np.arange(-10, 10).reshape(5, 4)
    _check_tables(_int8_plan(wi, -3, eb, m), *_expected(_f_hat(wi, -3), eb, m))


@pytest.mark.parametrize("m", MS)
def test_int8_plan_given_tap_exponents(m):
    wi = _int8_weights(41, 24, 40)
    e_f = -8
    rng = np.random.default_rng(42)
    # below and above the natural exponents (saturation, rounding to 0), with
    # the alignment shifts still within 62 bits
    eg = [int(v) for v in rng.integers(-28, 28, _ntap(m))]
    eb = _eb(m, 43)
    plan = _int8_plan(wi, e_f, eb, m, w_exp=eg)
    _check_tables(plan, *_expected(_f_hat(wi, e_f), eb, m, e_g=eg))
    # every tap 45 binades off: all Uq saturate, or all round to 0
    for k in (-45, 45):
        eg = [e_f + k] * _ntap(m)
        plan = _int8_plan(wi, e_f, eb, m, w_exp=eg)
        _check_tables(plan, *_expected(_f_hat(wi, e_f), eb, m, e_g=eg))


@pytest.mark.parametrize("m", MS)
def test_int8_plan_from_direct_quantization(m):
    """The chain the paper's formula describes: fp32 weights -> spatial int8
    f_hat (one power-of-two scale) -> Winograd plan -> convolution, equal to
    the oracle on the same f_hat."""
    n, cin, cout, h, w = 1, 48, 64, 16, 20
    x, f, b = workloads.random_case(44, n, cin, cout, h, w, signed=False)
    w_ohwi, e_f = W.direct_conv_quantize_weights(f)
    wi = np.ascontiguousarray(np.asarray(w_ohwi).transpose(0, 3, 1, 2))     # OHWI -> OIHW
    wq, e_or = direct.quantize_weights_pow2(f)
    assert e_f == e_or and (wi == wq).all()
    eb = tapwise.calibrate_input_exps(x, m=m)
    plan = _int8_plan(wi, e_f, eb, m, bias=b, out_shift=6)
    o = tapwise.make_plan(_f_hat(wi, e_f), eb, bias=b, out_shift=6, m=m)
    _check_tables(plan, o, 32 if tapwise.epilogue_bound(o) < 2 ** 31 else 64)
    assert (run_conv(plan, x, W.NHWC) == tapwise.conv_int8(x, o)).all()


def test_int8_plan_argument_errors():
    torch = torch_dev()
    wd = torch.zeros((2, 2, 3, 3), dtype=torch.int8, device="cuda")
    for bad_ef in (-127, 121):
        with pytest.raises(W.WinoError) as e:
            W.wino_f4_plan_int8(wd, bad_ef, [0] * 36)
        assert e.value.status == -1
    # e_f = -126 with small weights takes e_G below -126: out of range
    wi = np.ones((2, 2, 3, 3), np.int8)
    with pytest.raises(W.WinoError) as e:
        W.wino_f4_plan_int8(torch.from_numpy(wi).cuda(), -126, [0] * 36)
    assert e.value.status == -3
    with pytest.raises(ValueError):
        W.wino_f4_plan_int8(wd.float(), 0, [0] * 36)
