"""Pins of the CPU oracle against facts fixed by the paper and by mathematics
(no GPU).  Each test names what it pins and why a plausible slip in the oracle
(dropped term, wrong sign or index, transposed operand, wrong rounding) would
fail it."""
import itertools
import os
from fractions import Fraction as Fr

import numpy as np
import pytest

from oracle import direct, f4, quant, tapwise

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# transform matrices
# ---------------------------------------------------------------------------
def _parse_golden(path):
    mats, cur = {}, None
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        tok = line.split()
        if tok[0] == "matrix":
            cur = tok[1]
            mats[cur] = {"scale": Fr(1), "rows": []}
        elif tok[0] == "scale":
            mats[cur]["scale"] = Fr(tok[1])
        else:
            mats[cur]["rows"].append([Fr(t) for t in tok])
    return {k: [[v["scale"] * e for e in r] for r in v["rows"]] for k, v in mats.items()}


@pytest.mark.parametrize("fname,bt,g,at", [
    ("f4_matrices.txt", f4.BT4, f4.G4, f4.AT4),
    ("f2_matrices.txt", f4.BT2, f4.G2, f4.AT2),
])
def test_matrices_match_printed(fname, bt, g, at):
    """The oracle's matrices are the ones printed in Sec. II."""
    gold = _parse_golden(os.path.join(GOLDEN, fname))
    assert [[Fr(v) for v in r] for r in bt] == gold["BT"]
    assert [[Fr(v) for v in r] for r in g] == gold["G"]
    assert [[Fr(v) for v in r] for r in at] == gold["AT"]


def _identity_1d_holds(bt, g, at):
    """A^T[(G g) (.) (B^T d)] equals the correlation out[i] = sum_k d[i+k] g[k]
    for every pair of basis vectors (the map is bilinear, so this is the
    identity for all d, g)."""
    n_in, m = len(bt), len(at)
    for di in range(n_in):
        for gi in range(3):
            d = [Fr(int(k == di)) for k in range(n_in)]
            gv = [Fr(int(k == gi)) for k in range(3)]
            u = [sum(g[a][k] * gv[k] for k in range(3)) for a in range(n_in)]
            v = [sum(Fr(bt[a][k]) * d[k] for k in range(n_in)) for a in range(n_in)]
            y = [sum(Fr(at[i][a]) * u[a] * v[a] for a in range(n_in)) for i in range(m)]
            ref = [sum(d[i + k] * gv[k] for k in range(3)) for i in range(m)]
            if y != ref:
                return False
    return True


def test_f4_identity_1d_exact():
    assert _identity_1d_holds(f4.BT4, f4.G4, f4.AT4)


def test_f2_identity_1d_exact():
    assert _identity_1d_holds(f4.BT2, f4.G2, f4.AT2)


def test_f4_identity_2d_exact():
    """Eq. winograd on a 6x6 tile: Y = A^T[(G f G^T) (.) (B^T d B)]A equals the
    4x4 correlation of d with f, exactly, for all 36 x 9 basis pairs."""
    bt = np.array(f4.BT4, dtype=object)
    at = np.array(f4.AT4, dtype=object)
    g = np.array(f4.G4, dtype=object)
    for di, fi in itertools.product(range(36), range(9)):
        d = np.zeros((6, 6), dtype=object); d[divmod(di, 6)] = Fr(1)
        f = np.zeros((3, 3), dtype=object); f[divmod(fi, 3)] = Fr(1)
        u = g.dot(f).dot(g.T)
        v = bt.dot(d).dot(bt.T)
        y = at.dot(u * v).dot(at.T)
        ref = np.array([[sum(d[i + r, j + c] * f[r, c] for r in range(3) for c in range(3))
                         for j in range(4)] for i in range(4)], dtype=object)
        assert (y == ref).all(), (di, fi)


def test_identity_catches_single_entry_slips():
    """Planted mistakes (on the CPU): flipping the sign of, or zeroing, any one
    nonzero entry of B^T, G or A^T breaks the identity, so the identity tests
    above would catch a transcription slip anywhere."""
    def mutated(mat, i, j, fn):
        m = [list(r) for r in mat]
        m[i][j] = fn(m[i][j])
        return m
    for name in ("BT4", "G4", "AT4"):
        mat = getattr(f4, name)
        for i, row in enumerate(mat):
            for j, v in enumerate(row):
                if v == 0:
                    continue
                for fn in (lambda z: -z, lambda z: 0 * z):
                    args = {"BT4": f4.BT4, "G4": f4.G4, "AT4": f4.AT4}
                    args[name] = mutated(mat, i, j, fn)
                    assert not _identity_1d_holds(args["BT4"], args["G4"], args["AT4"]), (name, i, j)


def test_g24_is_24_times_g():
    for a in range(6):
        for k in range(3):
            assert Fr(f4.G4_INT[a][k], 24) == f4.G4[a][k]


def test_mac_reduction():
    """36 multiplies per 4x4 output tile and channel pair instead of 16*9 = 144
    (Sec. I: 4x for F4; 16 vs 36 for F2, 2.25x)."""
    assert len(f4.BT4) ** 2 * 4 == 16 * 9
    assert Fr(4 * 9, len(f4.BT2) ** 2) == Fr(9, 4)


# ---------------------------------------------------------------------------
# bit growth (Sec. II, Challenge I) -- exact integer bounds used to size the
# kernels' intermediates
# ---------------------------------------------------------------------------
def _box_max(coefs, lo, hi):
    pos = sum(c for c in coefs if c > 0)
    neg = -sum(c for c in coefs if c < 0)
    return max(pos * hi + neg * (-lo), pos * (-lo) + neg * hi)


def test_input_transform_bit_growth():
    bt = np.array(f4.BT4)
    kron = np.einsum("ar,bc->abrc", bt, bt).reshape(36, 36)
    assert max(_box_max(r, -128, 127) for r in kron) == 12768
    assert max(_box_max(r, 0, 127) for r in kron) == 8636
    # the row pass alone (one factor of B^T) stays within 10 * 128 = 1280
    assert max(_box_max(r, -128, 127) for r in bt) == 1278
    # both passes fit in int16 even with a rounding constant of 2^14 added
    assert 12768 + (1 << 14) < (1 << 15)
    # and the bound is attained: brute force over the extreme corners of one tap
    r0 = kron[0]
    d = np.where(r0 > 0, 127, np.where(r0 < 0, -128, 0)).reshape(6, 6)
    v = tapwise.input_transform(d[None])
    assert abs(int(v[0, 0, 0])) <= 12768


def test_output_transform_gain():
    at = np.array(f4.AT4)
    assert [int(np.abs(r).sum()) for r in at] == [5, 6, 10, 19]
    assert int(np.abs(np.einsum("ia,jb->ijab", at, at)).reshape(16, 36).sum(1).max()) == 361


# ---------------------------------------------------------------------------
# quantization rules (Eq. quant, Sec. III-B)
# ---------------------------------------------------------------------------
def test_round_half_up_ties():
    assert [quant.round_half_up(Fr(v, 2)) for v in (5, -5, 1, -1, 3, -3)] == [3, -2, 1, 0, 2, -1]
    assert quant.round_half_up(Fr(7, 3)) == 2 and quant.round_half_up(Fr(-7, 3)) == -2
    # integer shift formula agrees with the rational definition everywhere
    v = np.arange(-5000, 5001)
    for e in range(0, 9):
        ref = [quant.round_half_up(Fr(int(k), 2 ** e)) for k in v]
        assert quant.shift_round_int(v, e).tolist() == ref


def test_saturation_of_positive_max():
    """s = x_max / 2^(n-1): -x_max maps to -128, +x_max to 128 -> clamp 127."""
    xmax = Fr(37, 10)
    e = quant.cexp(xmax)          # scale 2^e >= xmax / 128
    s = Fr(2) ** e
    assert quant.quantize_exact(-xmax, e) >= -128
    xm = 128 * s                  # a value exactly at the power-of-two range
    assert quant.quantize_exact(xm, e) == 127
    assert quant.quantize_exact(-xm, e) == -128


def test_cexp_exact():
    assert quant.cexp(0) == 0
    assert quant.cexp(128) == 0
    assert quant.cexp(Fr(128) + Fr(1, 10 ** 30)) == 1
    assert quant.cexp(64) == -1
    assert quant.cexp(Fr(64) + Fr(1, 10 ** 30)) == 0
    assert quant.cexp(129) == 1 and quant.cexp(256) == 1 and quant.cexp(257) == 2
    assert quant.cexp(Fr(1, 2 ** 40)) == -47
    for a in [Fr(3, 7), Fr(1000), Fr(12768), Fr(1, 3)]:
        e = quant.cexp(a)
        assert a <= 128 * Fr(2) ** e and a > 128 * Fr(2) ** (e - 1)


# ---------------------------------------------------------------------------
# direct convolution: textbook definition, library routines, brute force
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed,n,cin,cout,h,w", [
    (0, 1, 1, 1, 1, 1), (1, 1, 2, 3, 3, 5), (2, 2, 3, 2, 9, 4), (3, 1, 3, 3, 2, 7)])
def test_direct_bruteforce(seed, n, cin, cout, h, w):
    rng = np.random.default_rng(seed)
    x = rng.integers(-128, 128, (n, cin, h, w))
    f = rng.integers(-128, 128, (cout, cin, 3, 3))
    bf = direct.conv_bruteforce(x.tolist(), f.tolist()).astype(np.int64)
    assert (direct.conv_int(x, f) == bf).all()
    assert np.allclose(direct.conv_f64(x, f), bf, rtol=0, atol=1e-9)


def test_direct_vs_scipy_and_torch():
    scipy_signal = pytest.importorskip("scipy.signal")
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    x = rng.normal(size=(2, 3, 11, 6))
    f = rng.normal(size=(4, 3, 3, 3))
    y = direct.conv_f64(x, f)
    ref = np.zeros_like(y)
    for b in range(2):
        for co in range(4):
            for ci in range(3):
                ref[b, co] += scipy_signal.correlate2d(x[b, ci], f[co, ci], mode="same")
    assert np.allclose(y, ref, atol=1e-12)
    yt = torch.nn.functional.conv2d(torch.from_numpy(x), torch.from_numpy(f), padding=1).numpy()
    assert np.allclose(y, yt, atol=1e-12)


def test_direct_int8_requant():
    rng = np.random.default_rng(9)
    x = rng.integers(-128, 128, (1, 2, 5, 5)).astype(np.int8)
    w = rng.integers(-128, 128, (3, 2, 3, 3)).astype(np.int8)
    b = rng.integers(-64, 65, 3)
    bf = direct.conv_bruteforce(x.astype(int).tolist(), w.astype(int).tolist())
    for s, relu in [(0, False), (7, False), (9, True)]:
        out = direct.conv_int8(x, w, b, s, relu)
        for idx in np.ndindex(out.shape):
            q = quant.clamp(quant.round_half_up(Fr(int(bf[idx]) + int(b[idx[1]]), 2 ** s)))
            assert out[idx] == (max(q, 0) if relu else q)


# ---------------------------------------------------------------------------
# float Winograd F4 (fp64) vs direct convolution
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("h,w", [(8, 8), (13, 6), (1, 1), (5, 3)])
def test_float_f4_equals_direct(h, w):
    rng = np.random.default_rng(h * 31 + w)
    x = rng.normal(size=(2, 5, h, w))
    f = rng.normal(size=(3, 5, 3, 3))
    yw = tapwise.conv_winograd_f64(x, f)
    yd = direct.conv_f64(x, f)
    assert np.abs(yw - yd).max() / np.abs(yd).max() <= 1e-4
    assert np.abs(yw - yd).max() / np.abs(yd).max() <= 1e-12


# ---------------------------------------------------------------------------
# plan: exact weight transform and tap quantization
# ---------------------------------------------------------------------------
def test_plan_uq_matches_rational_definition():
    """Uq and e_G from the integer-mantissa implementation equal a per-element
    evaluation with Fractions straight from the definition."""
    rng = np.random.default_rng(11)
    f = rng.normal(0, 0.2, (3, 2, 3, 3)).astype(np.float32)
    f[0, 0, 1, 1] = np.float32(1e-30)          # wide exponent spread
    f[1, 1] = 0.0                              # an all-zero kernel
    plan = tapwise.make_plan(f, [0] * 36)
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
        assert plan["e_g"][t] == quant.cexp(mx)
        for co in range(3):
            for ci in range(2):
                assert plan["uq"][t, ci, co] == quant.quantize_exact(U[co, ci, a, b], plan["e_g"][t])


def test_plan_ties_round_half_up():
    """Weights built so that U / 2^e_G lands exactly on half-integers."""
    f = np.zeros((1, 1, 3, 3), dtype=np.float32)
    f[0, 0, 1, 1] = np.float32(576 * 2.0 ** -6 * 3)     # U = 2^-6*3*outer(G24[:,1])
    e_g = [-6 + 1] * 36                                  # halves every tap value
    plan = tapwise.make_plan(f, [0] * 36, e_g=e_g)
    col = [row[1] for row in f4.G4_INT]
    for t in range(36):
        a, b = divmod(t, 6)
        v = Fr(3 * col[a] * col[b], 2)
        assert plan["uq"][t, 0, 0] == quant.clamp(quant.round_half_up(v))


# ---------------------------------------------------------------------------
# integer pipeline: two formulations, special cases, bounds
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed,n,cin,cout,h,w,relu", [
    (0, 1, 1, 1, 1, 1, False), (1, 1, 2, 3, 3, 5, True), (2, 2, 3, 2, 9, 4, False),
    (3, 1, 3, 1, 2, 7, True), (4, 1, 2, 2, 8, 8, False), (5, 1, 1, 2, 5, 6, False)])
def test_pipeline_batched_equals_naive(seed, n, cin, cout, h, w, relu):
    rng = np.random.default_rng(seed)
    x = rng.integers(-128, 128, (n, cin, h, w)).astype(np.int8)
    f = rng.normal(0, 0.3, (cout, cin, 3, 3)).astype(np.float32)
    b = rng.integers(-300, 301, cout)
    eb = [int(v) for v in rng.integers(0, 9, 36)]
    for s in (0, 5, 12):
        plan = tapwise.make_plan(f, eb, bias=b, out_shift=s, relu=relu)
        assert (tapwise.conv_int8(x, plan) == tapwise.conv_int8_naive(x, plan)).all()


def _lossless_case(seed, centre_only):
    rng = np.random.default_rng(seed)
    n, cin, cout, h, w = 2, 3, 4, 10, 7
    s = 5
    if centre_only:
        fint = np.zeros((cout, cin, 3, 3), dtype=np.int64)
        fint[:, :, 1, 1] = rng.integers(-1, 2, (cout, cin))
    else:
        fint = np.zeros((cout, cin, 3, 3), dtype=np.int64)
        fint[:, :, :2, :2] = rng.integers(-1, 2, (cout, cin, 2, 2))
    f = (576.0 * 2.0 ** -s * fint).astype(np.float32)
    return rng, n, cin, cout, h, w, s, fint, f


def test_lossless_equals_direct_uniform_scales():
    """Binary inputs (|V| <= 50, so e_B = 0 is exact) and weights
    f = 576 2^-s f_int with f_int on the 2x2 corner (|U 2^s| <= 64, so
    e_G = -s is exact): the integer pipeline must reproduce direct
    convolution exactly, Y 2^e_o = sum x f."""
    rng, n, cin, cout, h, w, s, fint, f = _lossless_case(1, centre_only=False)
    x = rng.integers(0, 2, (n, cin, h, w)).astype(np.int8)
    plan = tapwise.make_plan(f, [0] * 36, e_g=[-s] * 36)
    assert int(np.abs(plan["uq"]).max()) <= 64
    z = tapwise.prequant_output(x, plan)
    ref = 576 * direct.conv_int(x, fint)           # = 2^s * sum x f
    assert plan["e_o"] == -s
    assert (z == ref).all()


def test_lossless_equals_direct_unequal_shifts():
    """Unequal tap exponents: centre-only weights give U 2^s in {0, +-4, +-8,
    +-16}; per-tap e_G = -s + log2|U 2^s| makes Uq = +-1 exactly.  Inputs in
    {0, 8} with e_B[t] in {2, 3} are exact too.  The alignment shifts then
    differ across taps and the result must still equal direct convolution."""
    rng, n, cin, cout, h, w, s, fint, f = _lossless_case(2, centre_only=True)
    col = [row[1] for row in f4.G4_INT]            # [0, -4, 4, 2, -2, 0]
    e_g = []
    for t in range(36):
        m = abs(col[t // 6] * col[t % 6])
        e_g.append(-s + (m.bit_length() - 1 if m else 0))
    e_b = [int(v) for v in rng.integers(2, 4, 36)]
    x = (8 * rng.integers(0, 2, (n, cin, h, w))).astype(np.int8)
    plan = tapwise.make_plan(f, e_b, e_g=e_g)
    assert len(set(plan["sh"])) > 2
    z = tapwise.prequant_output(x, plan)
    ref = 576 * direct.conv_int(x, fint)
    scale = plan["e_o"] + s
    lhs = z * (2 ** scale) if scale >= 0 else z
    rhs = ref if scale >= 0 else ref * (2 ** -scale)
    assert (lhs == rhs).all()


def test_lossless_detects_dropped_alignment():
    """Planted mistake: with every alignment shift set to 0 the unequal-shift
    lossless case no longer equals direct convolution."""
    rng, n, cin, cout, h, w, s, fint, f = _lossless_case(2, centre_only=True)
    col = [row[1] for row in f4.G4_INT]
    e_g = [-s + (abs(col[t // 6] * col[t % 6]).bit_length() - 1 if col[t // 6] * col[t % 6] else 0)
           for t in range(36)]
    e_b = [int(v) for v in rng.integers(2, 4, 36)]
    x = (8 * rng.integers(0, 2, (n, cin, h, w))).astype(np.int8)
    plan = tapwise.make_plan(f, e_b, e_g=e_g)
    plan["sh"] = [0] * 36
    z = tapwise.prequant_output(x, plan)
    ref = 576 * direct.conv_int(x, fint)
    scale = plan["e_o"] + s
    assert not (z * 2 ** max(scale, 0) == ref * 2 ** max(-scale, 0)).all()


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_quantization_error_bound(seed):
    """Random data, calibrated scales: |Y 2^e_o - direct_fp64| obeys the
    analytic per-output bound of the two tap quantizations."""
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 128, (1, 6, 9, 11)).astype(np.int8)
    f = rng.normal(0, 0.15, (5, 6, 3, 3)).astype(np.float32)
    eb = tapwise.calibrate_input_exps(x)
    plan = tapwise.make_plan(f, eb)
    y = tapwise.prequant_output(x, plan).astype(np.float64) * 2.0 ** plan["e_o"]
    ref = direct.conv_f64(x, f.astype(np.float64))
    bound = tapwise.quantization_error_bound(x, f, plan, clamped_slack=True)
    err = np.abs(y - ref)
    assert (err <= bound * (1 + 1e-9) + 1e-9).all()
    # the approximation is meaningful: error well below the signal
    assert np.sqrt((err ** 2).mean()) < 0.5 * np.sqrt((ref ** 2).mean())


def test_error_bound_detects_wrong_tap_order():
    """Planted mistake: transposing the per-tap input exponents (tap a,b read
    as b,a) on asymmetric scales violates either exactness or the bound."""
    rng, n, cin, cout, h, w, s, fint, f = _lossless_case(3, centre_only=False)
    x = (8 * rng.integers(0, 2, (n, cin, h, w))).astype(np.int8)
    e_b = [3 if (t // 6) < (t % 6) else 2 for t in range(36)]   # |V| <= 400: exact, no clamp
    good = tapwise.make_plan(f, e_b, e_g=[-s] * 36)
    bad_eb = [e_b[(t % 6) * 6 + t // 6] for t in range(36)]
    bad = tapwise.make_plan(f, e_b, e_g=[-s] * 36)
    bad["e_b"] = bad_eb
    ref = 576 * direct.conv_int(x, fint)
    zg = tapwise.prequant_output(x, good) * 2 ** (good["e_o"] + s)
    zb = tapwise.prequant_output(x, bad) * 2 ** (bad["e_o"] + s)
    assert (zg == ref).all()
    assert not (zb == ref).all()


def test_calibration_minimal_and_safe():
    rng = np.random.default_rng(4)
    x = rng.integers(-128, 128, (2, 3, 10, 9)).astype(np.int8)
    amax = tapwise.input_tap_absmax(x)
    eb = tapwise.calibrate_input_exps(x)
    for t in range(36):
        assert amax[t] <= 128 * 2 ** eb[t]
        if eb[t] > 0:
            assert amax[t] > 128 * 2 ** (eb[t] - 1)
    f = rng.normal(0, 0.2, (4, 3, 3, 3)).astype(np.float32)
    plan = tapwise.make_plan(f, eb, bias=rng.integers(-64, 65, 4))
    s = tapwise.calibrate_out_shift(x, plan)
    z = tapwise.prequant_output(x, plan)
    assert np.abs(z).max() <= 128 * 2 ** s
    assert s == 0 or np.abs(z).max() > 128 * 2 ** (s - 1)


def test_epilogue_bound_dominates_actual_values():
    rng = np.random.default_rng(8)
    x = rng.integers(-128, 128, (1, 8, 8, 8)).astype(np.int8)
    f = rng.normal(0, 0.3, (3, 8, 3, 3)).astype(np.float32)
    eb = [int(v) for v in rng.integers(0, 8, 36)]
    plan = tapwise.make_plan(f, eb, bias=rng.integers(-64, 65, 3), out_shift=6)
    z = tapwise.prequant_output(x, plan)
    assert np.abs(z).max() + 32 <= tapwise.epilogue_bound(plan)
    # the bound is not absurdly loose for adversarial (all-extreme) inputs
    x2 = np.full((1, 8, 8, 8), -128, dtype=np.int8)
    assert tapwise.epilogue_bound(plan) < 2 ** 40


def test_empty_and_degenerate_shapes():
    f = np.zeros((2, 1, 3, 3), dtype=np.float32)
    plan = tapwise.make_plan(f, [0] * 36, bias=np.array([5, -7]), out_shift=1)
    assert plan["e_g"] == [0] * 36 and not plan["uq"].any()
    x = np.ones((1, 1, 1, 1), dtype=np.int8)
    y = tapwise.conv_int8(x, plan)
    assert y.tolist() == [[[[3]], [[-3]]]]       # R(5/2) = 3, R(-7/2) = -3
    x0 = np.zeros((0, 1, 4, 4), dtype=np.int8)
    assert tapwise.conv_int8(x0, plan).shape == (0, 2, 4, 4)
