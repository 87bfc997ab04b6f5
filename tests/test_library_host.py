"""CPU-side checks of the C-ABI library: it loads, exports every symbol the
header declares, its host plan arithmetic equals the oracle's, and invalid
arguments come back as status codes (no device work involved)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2209_12982_amd as W
import workloads
from oracle import direct, tapwise

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    try:
        return W.load_library()
    except W.LibraryNotBuilt:
        pytest.skip("library not built")


def _declared(header):
    hdr = open(os.path.join(ROOT, "include", header)).read()
    return re.findall(r"^\s*(?:wino_status|size_t|void|const char\*)\s+(\w+)\s*\(", hdr, re.M)


def test_exports_every_declared_symbol():
    """The method's header and the binding's EXPORTS list the same functions,
    the measurement header and PROBE_EXPORTS likewise, the two sets are
    disjoint, every header under include/ is one of the two, and the built
    library resolves every name."""
    lib = _lib()
    assert sorted(os.listdir(os.path.join(ROOT, "include"))) == ["winof4.h", "winof4_probe.h"]
    method, probe = _declared("winof4.h"), _declared("winof4_probe.h")
    assert len(method) >= 12 and probe
    assert sorted(method) == sorted(W.binding.EXPORTS)
    assert sorted(probe) == sorted(W.binding.PROBE_EXPORTS)
    assert not set(method) & set(probe)
    for name in method + probe:
        assert hasattr(lib, name), name


@pytest.mark.parametrize("name", ["C1", "C2", "C3"])
def test_plan_tables_match_oracle_on_configs(name):
    _lib()
    x, layers = workloads.generate(name)
    for f, b, spec in layers:
        eb = [int(v) for v in np.random.default_rng(spec.cin).integers(0, 8, 36)]
        for out_shift in (0, 11):
            c = W.wino_f4_plan_tables(f, eb, bias=b, out_shift=out_shift)
            o = tapwise.make_plan(f, eb, bias=b, out_shift=out_shift)
            assert c["e_g"] == o["e_g"] and c["sh"] == o["sh"] and c["e_o"] == o["e_o"]
            assert (c["uq"] == o["uq"]).all()
            bits = 32 if tapwise.epilogue_bound(o) < 2 ** 31 else 64
            assert c["epilogue_bits"] == bits


@pytest.mark.slow
def test_plan_tables_match_oracle_c5():
    _lib()
    x, layers = workloads.generate("C5")
    f, b, spec = layers[0]
    eb = [5, 5, 5, 4, 4, 5] * 6
    c = W.wino_f4_plan_tables(f, eb, bias=b, out_shift=11)
    o = tapwise.make_plan(f, eb, bias=b, out_shift=11)
    assert c["e_g"] == o["e_g"] and c["sh"] == o["sh"] and c["e_o"] == o["e_o"]
    assert (c["uq"] == o["uq"]).all()


def test_plan_tables_adversarial():
    """Exact ties, tap maxima exactly at 128 * 2^k, zero taps, tiny and huge
    magnitudes, explicit exponents."""
    _lib()
    rng = np.random.default_rng(3)
    cases = []
    f = np.zeros((2, 3, 3, 3), np.float32)
    f[0, 0, 1, 1] = 576 * 2.0 ** -6 * 3             # half-integer taps under e_G = -5
    f[1, 2] = 1.0
    cases.append((f, [-5] * 36))
    f2 = np.zeros((3, 2, 3, 3), np.float32)
    f2[:, :, :2, :2] = 576 * 2.0 ** -3 * rng.integers(-1, 2, (3, 2, 2, 2))   # max exactly 64*2^-3*...
    cases.append((f2, None))
    f3 = rng.normal(0, 1, (4, 3, 3, 3)).astype(np.float32)
    f3[0, 0, 0, 0] = np.float32(1e-38)
    f3[1, 1, 2, 2] = np.float32(3e4)
    cases.append((f3, None))
    cases.append((np.zeros((1, 1, 3, 3), np.float32), None))
    f4 = np.full((2, 2, 3, 3), -0.25, np.float32)
    cases.append((f4, None))
    for f, eg in cases:
        eb = [int(v) for v in rng.integers(0, 16, 36)]
        c = W.wino_f4_plan_tables(f, eb, w_exp=eg, out_shift=3)
        o = tapwise.make_plan(f, eb, e_g=eg, out_shift=3)
        assert c["e_g"] == o["e_g"] and c["sh"] == o["sh"] and c["e_o"] == o["e_o"]
        assert (c["uq"] == o["uq"]).all()


@pytest.mark.parametrize("name", ["C1", "C2", "C3"])
def test_f2_plan_tables_match_oracle_on_configs(name):
    _lib()
    x, layers = workloads.generate(name)
    for f, b, spec in layers:
        eb = [int(v) for v in np.random.default_rng(spec.cin + 1).integers(0, 4, 16)]
        for out_shift in (0, 9):
            c = W.wino_f2_plan_tables(f, eb, bias=b, out_shift=out_shift)
            o = tapwise.make_plan(f, eb, bias=b, out_shift=out_shift, m=2)
            assert c["e_g"] == o["e_g"] and c["sh"] == o["sh"] and c["e_o"] == o["e_o"]
            assert (c["uq"] == o["uq"]).all()
            bits = 32 if tapwise.epilogue_bound(o) < 2 ** 31 else 64
            assert c["epilogue_bits"] == bits


def test_f2_plan_tables_adversarial():
    """F2 (G = Gint / 2): exact ties, maxima exactly at 128 * 2^k, zero taps,
    extreme magnitudes, explicit exponents."""
    _lib()
    rng = np.random.default_rng(5)
    cases = []
    f = np.zeros((2, 3, 3, 3), np.float32)
    f[0, 0, 1, 1] = 4 * 2.0 ** -6 * 3              # U = 3 * 2^-6 * outer(Gint[:,1])
    f[1, 2] = 1.0
    cases.append((f, [-5] * 16))
    f2 = np.zeros((3, 2, 3, 3), np.float32)
    f2[:, :, 0, 0] = 4 * 2.0 ** -3 * 32 * rng.integers(-1, 2, (3, 2))   # |U| reaches 128 * 2^k
    cases.append((f2, None))
    f3 = rng.normal(0, 1, (4, 3, 3, 3)).astype(np.float32)
    f3[0, 0, 0, 0] = np.float32(1e-38)
    f3[1, 1, 2, 2] = np.float32(3e4)
    cases.append((f3, None))
    cases.append((np.zeros((1, 1, 3, 3), np.float32), None))
    for f, eg in cases:
        eb = [int(v) for v in rng.integers(0, 16, 16)]
        c = W.wino_f2_plan_tables(f, eb, w_exp=eg, out_shift=3)
        o = tapwise.make_plan(f, eb, e_g=eg, out_shift=3, m=2)
        assert c["e_g"] == o["e_g"] and c["sh"] == o["sh"] and c["e_o"] == o["e_o"]
        assert (c["uq"] == o["uq"]).all()


def test_select_algorithm_on_configs():
    """The per-layer rule picks what was measured fastest on MI355X for every
    layer of C1-C5 (host only: with no device the rule assumes 256 CUs)."""
    _lib()
    want = {"C1": [W.ALGO_DIRECT], "C2": [W.ALGO_F2], "C3": [W.ALGO_F2] * 4, "C4": [W.ALGO_F4], "C5": [W.ALGO_F4]}
    for name, algos in want.items():
        wl = workloads.WORKLOADS[name]
        got = [W.wino_select_algorithm(wl.n, s.cin, s.cout, s.h, s.w) for s in wl.layers]
        assert got == algos, name
    # NCHW: the direct convolution there is the simple kernel, so small layers take F2
    wl = workloads.WORKLOADS["C1"]
    s = wl.layers[0]
    assert W.wino_select_algorithm(wl.n, s.cin, s.cout, s.h, s.w, W.NCHW) == W.ALGO_F2
    assert W.wino_select_algorithm(8, 64, 64, 56, 56, W.NCHW) == W.ALGO_F2
    with pytest.raises(W.WinoError):
        W.wino_select_algorithm(1, 0, 4, 8, 8)
    with pytest.raises(W.WinoError):
        W.wino_select_algorithm(1, 4, 4, 8, 8, 7)


def test_direct_weight_quantization_matches_oracle():
    _lib()
    rng = np.random.default_rng(4)
    f = rng.normal(0, 0.2, (5, 7, 3, 3)).astype(np.float32)
    f[0, 0, 0, 0] = 0.5 * 2.0 ** -3            # tie at the scale chosen below
    w, e = W.direct_conv_quantize_weights(f)
    wr, er = direct.quantize_weights_pow2(f)
    assert e == er and (w == wr.transpose(0, 2, 3, 1)).all()


def test_invalid_arguments_return_status():
    lib = _lib()
    P = ctypes.c_void_p
    assert lib.wino_f4_conv_int8(None, None, None, 1, 4, 4, 0, 0, None, 0, None) == -1
    assert lib.wino_f4_workspace_bytes(None, 1, 4, 4, 0) == 0
    assert lib.wino_f4_plan_info(None, None, None, None, None, None, None, None) == -1
    assert lib.wino_f4_plan_set_tap_kernel(None, 0) == -1
    assert lib.direct_conv_int8(None, None, None, None, 1, 1, 1, 1, 1, 0, 0, 0, None) == -1
    x = np.zeros(16, np.int8)
    # bad layout / shift / relu / sizes are rejected before any launch
    assert lib.direct_conv_int8(x.ctypes.data, x.ctypes.data, None, x.ctypes.data, 1, 1, 1, 4, 4, 7, 0, 0, None) == -1
    assert lib.direct_conv_int8(x.ctypes.data, x.ctypes.data, None, x.ctypes.data, 1, 1, 1, 4, 4, 0, 40, 0, None) == -1
    assert lib.direct_conv_int8(x.ctypes.data, x.ctypes.data, None, x.ctypes.data, 1, 9000, 1, 4, 4, 0, 0, 0, None) == -2
    assert lib.wino_f4_calibrate_input(x.ctypes.data, -1, 1, 4, 4, 0, None, None, None) == -1
    f = np.zeros((1, 1, 3, 3), np.float32)
    eb = np.zeros(36, np.int8)
    bad = eb.copy(); bad[3] = 16
    h = P()
    assert lib.wino_f4_plan(None, f.ctypes.data, 1, 1, eb.ctypes.data, None, None, 0, 0, None) == -1
    assert lib.wino_f4_plan(ctypes.byref(h), f.ctypes.data, 1, 1, bad.ctypes.data, None, None, 0, 0, None) == -1
    assert h.value is None
    assert lib.wino_f4_plan(ctypes.byref(h), f.ctypes.data, 1, 1, eb.ctypes.data, None, None, 63, 0, None) == -1
    assert lib.wino_f4_plan(ctypes.byref(h), f.ctypes.data, 0, 1, eb.ctypes.data, None, None, 0, 0, None) == -1
    fn = f.copy(); fn[0, 0, 0, 0] = np.nan
    assert lib.wino_f4_plan(ctypes.byref(h), fn.ctypes.data, 1, 1, eb.ctypes.data, None, None, 0, 0, None) == -1
    # alignment shifts beyond what any epilogue holds
    eg = np.zeros(36, np.int8); eg[0] = 100; eg[1] = -100
    assert lib.wino_f4_plan_tables(f.ctypes.data, 1, 1, eb.ctypes.data, eg.ctypes.data, None, 0,
                                   None, None, None, None, None) == -3
    # the fp32 reference stage validates before any launch too
    fw = np.zeros(9, np.float32)
    yf = np.zeros(16, np.float32)
    assert lib.wino_f4_conv_float(None, fw.ctypes.data, yf.ctypes.data, 1, 1, 1, 4, 4, 0, None) == -1
    assert lib.wino_f4_conv_float(x.ctypes.data, fw.ctypes.data, yf.ctypes.data, 1, 0, 1, 4, 4, 0, None) == -1
    assert lib.wino_f4_conv_float(x.ctypes.data, fw.ctypes.data, yf.ctypes.data, 1, 1, 1, 4, 4, 7, None) == -1
    assert lib.wino_f4_conv_float(x.ctypes.data, fw.ctypes.data, yf.ctypes.data, 1, 70000, 1, 4, 4, 0, None) == -2
    # the matrix-core probe checks its arguments before launching
    ops = ctypes.c_int64()
    assert lib.wino_probe_mfma_int8(7, 10, 1, x.ctypes.data, ctypes.byref(ops), None) == -1
    assert lib.wino_probe_mfma_int8(16, 0, 1, x.ctypes.data, ctypes.byref(ops), None) == -1
    assert lib.wino_probe_mfma_int8(32, 10, 1, None, ctypes.byref(ops), None) == -1
    lib.wino_f4_plan_destroy(None)
    assert W.wino_strerror(-5).startswith("workspace")


def test_epilogue_width_decision():
    """The host bound picks 32 bits for calibrated data and 64 bits when the
    alignment shifts are large, as the oracle's bound says."""
    _lib()
    x, f, b = workloads.random_case(6, 1, 20, 24, 11, 10, signed=True)
    eb = [0] * 36
    eb[35], eb[0] = 15, 14
    c = W.wino_f4_plan_tables(f, eb, bias=b, out_shift=20)
    o = tapwise.make_plan(f, eb, bias=b, out_shift=20)
    assert c["epilogue_bits"] == 64 and tapwise.epilogue_bound(o) >= 2 ** 31
