"""Tap-wise quantized integer Winograd F(4x4, 3x3) and F(2x2, 3x3) (Sec. II
matrices; Sec. III, Eq. winograd, Eq. quant, the rearranged tap-wise scheme,
and power-of-two scales of Sec. III-B), plus the float64 Winograd algorithm
they approximate.  Every function takes the F4 transform by default; a plan
records its output tile size m (4 or 2) and the functions that take a plan
follow it.

Definition followed (one output channel co, one 4x4 tile):

  Y = A^T ( S_BG (.) sum_ci  q(B^T d_ci B (/) S_B) (.) q(G f_co,ci G^T (/) S_G) ) A

with S_B = 2^e_B and S_G = 2^e_G per tap (element-wise), S_BG = S_B (.) S_G,
and q the int8 quantizer of Eq. quant (round half up, clamp [-128, 127]).
The int8 x int8 products are accumulated over ci as integers and the tap
scale is applied once, before the back transform.  S_BG is realised without
any rounding: every tap is aligned to the smallest exponent
e_o = min_t (e_B[t] + e_G[t]) by an exact factor 2^sh[t], sh = e_B + e_G - e_o,
so Y is an exact integer and the real-valued output is Y * 2^e_o.  The output
is then requantised: z = Y + bias (bias in units of 2^e_o),
out = clamp(R(z / 2^out_shift)), optionally max(out, 0).

Offline (the plan): U = G f G^T is computed exactly (weights are fp32, hence
dyadic rationals, and G = G24 / 24 with G24 integral), e_G[t] = cexp(max over
(co, ci) of |U_t|) unless given, and Uq = q(U / 2^e_G).

Input tiles are 6x6 windows at stride 4 over the input padded by one zero
pixel on each side; ceil(H/4) x ceil(W/4) tiles are computed and outputs
outside the image are discarded (zero padding to a multiple of 4, Sec. V).
For F(2x2, 3x3) the same holds with 4x4 windows at stride 2, 16 taps, and
G = G2int / 2 (so U = unum * 2^p / 4).

int8/10 (Sec. V): with bits = 10 the Winograd-domain integers Vq and Uq are
quantized to 10 bits ([-512, 511], scale exponents from 2^9 instead of 2^7)
while the spatial input and output stay int8; a plan
records its ``bits`` and every function that takes a plan follows it.
"""
from fractions import Fraction

import numpy as np

from . import f4, quant



class Spec:
    """One Winograd transform F(m x m, 3 x 3): input tiles n x n (n = m + 2)
    at stride m, n^2 taps, B^T (n x n), A^T (m x n) and G = Gint / den with
    Gint integral (n x 3)."""

    def __init__(self, m, bt, at, g, den):
        self.m, self.n = m, m + 2
        self.ntap = self.n * self.n
        self.BT = f4.as_int_array(bt)
        self.AT = f4.as_int_array(at)
        self.Gint = f4.g_times(den, g)
        self.den = den
        self.bt, self.at, self.g = bt, at, g      # exact (rational) entries


F4 = Spec(4, f4.BT4, f4.AT4, f4.G4, f4.G4_DEN)
F2 = Spec(2, f4.BT2, f4.AT2, f4.G2, 2)
SPECS = {4: F4, 2: F2}

# the F4 names used throughout (and by the tests)
NTAP = F4.ntap
BT = F4.BT             # 6x6
AT = F4.AT             # 4x6
G24 = F4.Gint          # 6x3 integers, G = G24 / 24


def spec_of(plan):
    return SPECS[plan.get("m", 4)]


# ---------------------------------------------------------------------------
# offline plan
# ---------------------------------------------------------------------------
def weight_transform_exact(f, spec=F4):
    """Exact U = G f G^T for fp32 weights f [cout, cin, 3, 3].

    Returns (unum, p): unum is an object array of Python ints with shape
    [cout, cin, n, n] and U = unum * 2^p / den^2 exactly (den^2 = 576 for
    F4, 4 for F2).
    """
    f = np.asarray(f, dtype=np.float32)
    cout, cin = f.shape[:2]
    assert f.shape == (cout, cin, 3, 3)
    mant, ex = np.frexp(f.astype(np.float64))        # f = mant * 2^ex
    m = (mant * float(1 << 24)).astype(np.int64)      # exact: 24-bit significand
    k = ex.astype(np.int64) - 24                      # f = m * 2^k
    nz = m != 0
    p = int(k[nz].min()) if nz.any() else 0
    F = np.empty(f.shape, dtype=object)
    mflat, kflat, Fflat = m.ravel(), k.ravel(), F.reshape(-1)
    for i in range(mflat.size):
        Fflat[i] = int(mflat[i]) << int(kflat[i] - p) if mflat[i] != 0 else 0
    g = np.array(spec.Gint, dtype=object)             # n x 3
    unum = np.matmul(np.matmul(g, F), g.T)            # [cout, cin, n, n]
    return unum, p


def _u_abs_max_per_tap(unum, p, spec=F4):
    """max over (co, ci) of |U_t| for every tap, as exact Fractions."""
    out = []
    flat = unum.reshape(-1, spec.ntap)
    d2 = spec.den * spec.den
    for t in range(spec.ntap):
        mx = max((abs(v) for v in flat[:, t]), default=0)
        out.append(Fraction(mx) * Fraction(2) ** p / d2)
    return out


def _quantize_unum(unum, p, e_g, spec=F4, bits=8):
    """Uq = clamp(R(U / 2^e_G)) with U = unum * 2^p / den^2, per tap:
    R(v) = floor(v + 1/2) = floor((2 unum 2^(p - e_G) + den^2) / (2 den^2))."""
    cout, cin = unum.shape[:2]
    flat = unum.reshape(cout, cin, spec.ntap)
    d2 = spec.den * spec.den
    uq = np.zeros((cout, cin, spec.ntap), dtype=np.int64)
    for t in range(spec.ntap):
        s = p - e_g[t]
        col = flat[:, :, t]
        if s >= 0:
            num = 2 * col * (1 << s) + d2
            den = 2 * d2
        else:
            num = 2 * col + d2 * (1 << -s)
            den = 2 * d2 * (1 << -s)
        q = num // den                                 # floor division
        uq[:, :, t] = np.clip(q.astype(np.int64) if q.dtype != object
                              else np.array([[int(v) for v in row] for row in q], dtype=np.int64),
                              *quant.qrange(bits))
    return uq


def make_plan(f, e_b, e_g=None, bias=None, out_shift=0, relu=False, m=4, bits=8):
    """The offline step: returns a dict with m, bits, e_B, e_G, e, e_o, sh, Uq
    [ntap, cin, cout] (tap-major GEMM operand), bias [cout], out_shift, relu.
    ``bits`` is the width of the Winograd-domain integers (Vq and Uq): 8, or
    10 for the int8/10 variant of Sec. V (spatial input and output stay int8)."""
    spec = SPECS[m]
    f = np.asarray(f, dtype=np.float32)
    cout, cin = f.shape[:2]
    e_b = [int(v) for v in e_b]
    assert len(e_b) == spec.ntap
    unum, p = weight_transform_exact(f, spec)
    if e_g is None:
        e_g = [quant.cexp(a, bits) for a in _u_abs_max_per_tap(unum, p, spec)]
    else:
        e_g = [int(v) for v in e_g]
        assert len(e_g) == spec.ntap
    uq = _quantize_unum(unum, p, e_g, spec, bits)     # [cout, cin, ntap]
    e = [e_b[t] + e_g[t] for t in range(spec.ntap)]
    e_o = min(e)
    sh = [e[t] - e_o for t in range(spec.ntap)]
    if bias is None:
        bias = np.zeros(cout, dtype=np.int64)
    return dict(m=m, bits=bits, cin=cin, cout=cout, e_b=e_b, e_g=e_g, e=e, e_o=e_o, sh=sh,
                uq=np.ascontiguousarray(uq.transpose(2, 1, 0)),   # [ntap, cin, cout]
                bias=np.asarray(bias, dtype=np.int64).copy(),
                out_shift=int(out_shift), relu=bool(relu))


# ---------------------------------------------------------------------------
# online integer pipeline, batched formulation
# ---------------------------------------------------------------------------
def tile_grid(h, w, m=4):
    return -(-h // m), -(-w // m)


def input_tiles(x, spec=F4):
    """d[n, ci, ty, tx, r, c] = x[n, ci, m ty + r - 1, m tx + c - 1], zero
    outside the image (r, c < m + 2)."""
    x = np.asarray(x, dtype=np.int64)
    n, cin, h, w = x.shape
    m, k = spec.m, spec.n
    th, tw = tile_grid(h, w, m)
    p = np.zeros((n, cin, m * th + 2, m * tw + 2), dtype=np.int64)
    p[:, :, 1:h + 1, 1:w + 1] = x
    d = np.zeros((n, cin, th, tw, k, k), dtype=np.int64)
    for r in range(k):
        for c in range(k):
            d[:, :, :, :, r, c] = p[:, :, r:r + m * th:m, c:c + m * tw:m]
    return d


def input_transform(d, spec=F4):
    """V = B^T d B on every tile (exact int64)."""
    return np.einsum("ar,...rc,bc->...ab", spec.BT, d, spec.BT)


def quantize_input_taps(v, e_b, spec=F4, bits=8):
    """Vq[..., a, b] = clamp(R(V[..., a, b] / 2^e_B[n a + b])) to bits-wide integers."""
    vq = np.empty_like(v)
    for t in range(spec.ntap):
        a, b = divmod(t, spec.n)
        vq[..., a, b] = quant.clamp_bits(quant.shift_round_int(v[..., a, b], e_b[t]), bits)
    return vq


def tap_major(vq, spec=F4):
    """[n, cin, th, tw, k, k] -> [ntap, T, cin] with tile index (n*th + ty)*tw + tx."""
    n, cin, th, tw = vq.shape[:4]
    return np.ascontiguousarray(vq.reshape(n, cin, th * tw, spec.ntap).transpose(3, 0, 2, 1)
                                .reshape(spec.ntap, n * th * tw, cin))


def tap_gemm(vq_tm, uq):
    """M[t] = Vq[t] @ Uq[t]: [ntap, T, cin] x [ntap, cin, cout] -> int64 [ntap, T, cout].
    Evaluated with float64 BLAS, exact because every partial sum is an
    integer of magnitude <= 2^18 * cin < 2^53 (operands of at most 10 bits)."""
    cin = vq_tm.shape[2]
    assert cin < (1 << 38)
    m = np.matmul(vq_tm.astype(np.float64), uq.astype(np.float64))
    return m.astype(np.int64)


def output_transform(m, sh, spec=F4):
    """Y = A^T (M (.) 2^sh) A.  m [ntap, T, cout] -> Y [T, cout, m, m] (int64).
    The caller guarantees no int64 overflow (checked here)."""
    nt, cout = m.shape[1:]
    k = spec.n
    mm = np.empty_like(m)
    for t in range(spec.ntap):
        assert sh[t] < 40
        mm[t] = m[t] * (np.int64(1) << np.int64(sh[t]))
    assert np.abs(mm).max(initial=0) < (1 << 50)
    mk = mm.reshape(k, k, nt, cout).transpose(2, 3, 0, 1)        # [T, cout, k, k]
    return np.einsum("ia,...ab,jb->...ij", spec.AT, mk, spec.AT)


def assemble(yt, n, h, w, spec=F4):
    """[T, cout, m, m] tiles -> [n, cout, h, w], dropping out-of-image rows/cols."""
    m = spec.m
    th, tw = tile_grid(h, w, m)
    cout = yt.shape[1]
    y = yt.reshape(n, th, tw, cout, m, m).transpose(0, 3, 1, 4, 2, 5)
    return y.reshape(n, cout, m * th, m * tw)[:, :, :h, :w]


def prequant_output(x, plan):
    """z = Y + bias on in-image outputs, [n, cout, h, w] int64."""
    spec = spec_of(plan)
    x = np.asarray(x)
    n, cin, h, w = x.shape
    assert cin == plan["cin"]
    v = input_transform(input_tiles(x, spec), spec)
    vq = quantize_input_taps(v, plan["e_b"], spec, plan.get("bits", 8))
    m = tap_gemm(tap_major(vq, spec), plan["uq"])
    y = assemble(output_transform(m, plan["sh"], spec), n, h, w, spec)
    return y + plan["bias"][None, :, None, None]


def requant(z, out_shift, relu):
    out = quant.clamp_int8(quant.shift_round_int(z, out_shift))
    if relu:
        out = np.maximum(out, 0)
    return out.astype(np.int8)


def conv_int8(x, plan):
    """The whole online path on int8 NCHW input: int8 NCHW output."""
    return requant(prequant_output(x, plan), plan["out_shift"], plan["relu"])


def input_taps_quantized(x, e_b, m=4, bits=8):
    """Vq in tap-major layout [ntap, T, cin] (what the input-transform stage emits)."""
    spec = SPECS[m]
    return tap_major(quantize_input_taps(input_transform(input_tiles(x, spec), spec), e_b, spec, bits), spec)


# ---------------------------------------------------------------------------
# online integer pipeline, naive per-tile formulation (independent spelling)
# ---------------------------------------------------------------------------
def conv_int8_naive(x, plan):
    """Same definition, written as scalar loops over tiles, channels and taps
    with Python integers.  Only for tiny shapes."""
    spec = spec_of(plan)
    mt, k, ntap = spec.m, spec.n, spec.ntap
    x = np.asarray(x, dtype=np.int64)
    n, cin, h, w = x.shape
    cout = plan["cout"]
    th, tw = tile_grid(h, w, mt)
    uq = plan["uq"]
    bt = spec.bt
    at = spec.at
    out = np.zeros((n, cout, h, w), dtype=np.int8)

    def px(b, ci, r, c):
        return int(x[b, ci, r, c]) if 0 <= r < h and 0 <= c < w else 0

    for b in range(n):
        for ty in range(th):
            for tx in range(tw):
                vq = []                                   # vq[ci][t]
                for ci in range(cin):
                    d = [[px(b, ci, mt * ty + r - 1, mt * tx + c - 1) for c in range(k)]
                         for r in range(k)]
                    row = []
                    for t in range(ntap):
                        a, bb = divmod(t, k)
                        v = sum(bt[a][r] * d[r][c] * bt[bb][c]
                                for r in range(k) for c in range(k))
                        q = quant.clamp(quant.round_half_up(Fraction(v, 2 ** plan["e_b"][t])),
                                        *quant.qrange(plan.get("bits", 8)))
                        row.append(q)
                    vq.append(row)
                for co in range(cout):
                    msh = []
                    for t in range(ntap):
                        acc = sum(vq[ci][t] * int(uq[t, ci, co]) for ci in range(cin))
                        msh.append(acc * 2 ** plan["sh"][t])
                    for i in range(mt):
                        for j in range(mt):
                            yy, xx = mt * ty + i, mt * tx + j
                            if yy >= h or xx >= w:
                                continue
                            val = sum(at[i][t // k] * at[j][t % k] * msh[t] for t in range(ntap))
                            z = val + int(plan["bias"][co])
                            q = quant.clamp(quant.round_half_up(Fraction(z, 2 ** plan["out_shift"])))
                            if plan["relu"]:
                                q = max(q, 0)
                            out[b, co, yy, xx] = q
    return out


# ---------------------------------------------------------------------------
# calibration (max-abs, power-of-two; Sec. III quantization + Sec. III-B)
# ---------------------------------------------------------------------------
EB_MAX = 15
OUT_SHIFT_MAX = 62


def input_tap_absmax(x, m=4):
    spec = SPECS[m]
    v = input_transform(input_tiles(x, spec), spec)
    return [int(np.abs(v[..., t // spec.n, t % spec.n]).max(initial=0)) for t in range(spec.ntap)]


def calibrate_input_exps(x, m=4, bits=8):
    """e_B[t] = max(0, cexp(max over tiles and channels of |V_t|)), <= 15, for
    bits-wide input taps."""
    return [min(EB_MAX, max(0, quant.cexp(a, bits))) for a in input_tap_absmax(x, m)]


def calibrate_out_shift(x, plan):
    """out_shift = max(0, cexp(max |Y + bias|)) over in-image outputs."""
    z = prequant_output(x, plan)
    return min(OUT_SHIFT_MAX, max(0, quant.cexp(int(np.abs(z).max(initial=0)))))


# ---------------------------------------------------------------------------
# analytic bounds
# ---------------------------------------------------------------------------
def epilogue_bound(plan):
    """Upper bound on |every partial sum of the output transform| plus bias
    and rounding constant:
      max_co max_ij sum_t |A^T[i,a] A^T[j,b]| 2^sh[t] vmax sum_ci |Uq[t,ci,co]|
      + max|bias| + (2^(out_shift-1) if out_shift > 0), with vmax = 2^(bits-1)
      the largest |Vq| (128 for int8)."""
    spec = spec_of(plan)
    vmax = 1 << (plan.get("bits", 8) - 1)
    uq = plan["uq"]
    s = np.abs(uq).sum(axis=1)                                 # [ntap, cout]
    best = 0
    for co in range(plan["cout"]):
        for i in range(spec.m):
            for j in range(spec.m):
                tot = 0
                for t in range(spec.ntap):
                    a, b = divmod(t, spec.n)
                    tot += (abs(int(spec.AT[i, a]) * int(spec.AT[j, b])) * (1 << plan["sh"][t]) * vmax
                            * int(s[t, co]))
                best = max(best, tot)
    rnd = (1 << (plan["out_shift"] - 1)) if plan["out_shift"] > 0 else 0
    return best + int(np.abs(plan["bias"]).max(initial=0)) + rnd


def quantization_error_bound(x, f, plan, clamped_slack=False):
    """Per-output bound on |Y * 2^e_o - direct_fp64(x, f)| (before bias and
    requant): sum_t |A^T[i,a] A^T[j,b]| sum_ci (dB |U_t| + |V_t| dG + dB dG)
    with dB = 2^(e_B-1), dG = 2^(e_G-1) (2^e with ``clamped_slack`` to also
    cover the single +128 -> 127 saturation).  Returns [n, cout, h, w] float64."""
    spec = spec_of(plan)
    x = np.asarray(x)
    n, cin, h, w = x.shape
    unum, p = weight_transform_exact(f, spec)
    d2 = spec.den * spec.den
    u_abs = np.abs(np.array([[[float(Fraction(int(v)) * Fraction(2) ** p / d2) for v in blk.ravel()]
                               for blk in row] for row in unum]))           # [cout, cin, ntap]
    v = input_transform(input_tiles(x, spec), spec)                          # [n,cin,th,tw,k,k]
    v_abs = np.abs(tap_major(v, spec)).astype(np.float64)                    # [ntap, T, cin]
    k = 0 if clamped_slack else 1
    db = np.array([2.0 ** (plan["e_b"][t] - k) for t in range(spec.ntap)])
    dg = np.array([2.0 ** (plan["e_g"][t] - k) for t in range(spec.ntap)])
    ua = u_abs.transpose(2, 1, 0)                                            # [ntap, cin, cout]
    err = (db[:, None, None] * ua.sum(axis=1)[:, None, :]
           + dg[:, None, None] * v_abs.sum(axis=2)[:, :, None]
           + (db * dg)[:, None, None] * cin)                                # [ntap, T, cout]
    coef = np.abs(np.einsum("ia,jb->ijab", spec.AT, spec.AT)).reshape(spec.m, spec.m, spec.ntap).astype(np.float64)
    bt = np.einsum("ijt,tkc->kcij", coef, err)                               # [T, cout, m, m]
    return assemble(bt, n, h, w, spec)


# ---------------------------------------------------------------------------
# float64 Winograd F(m x m, 3 x 3) without quantization (Eq. winograd)
# ---------------------------------------------------------------------------
def conv_winograd_f64(x, f, m=4):
    spec = SPECS[m]
    k = spec.n
    x = np.asarray(x, dtype=np.float64)
    f = np.asarray(f, dtype=np.float64)
    n, cin, h, w = x.shape
    g = f4.as_f64_array(spec.g)
    bt = spec.BT.astype(np.float64)
    at = spec.AT.astype(np.float64)
    u = np.einsum("ar,oirc,bc->oiab", g, f, g)                    # [cout, cin, k, k]
    th, tw = tile_grid(h, w, m)
    p = np.zeros((n, cin, m * th + 2, m * tw + 2))
    p[:, :, 1:h + 1, 1:w + 1] = x
    d = np.zeros((n, cin, th, tw, k, k))
    for r in range(k):
        for c in range(k):
            d[:, :, :, :, r, c] = p[:, :, r:r + m * th:m, c:c + m * tw:m]
    v = np.einsum("ar,niyxrc,bc->niyxab", bt, d, bt)
    mm = np.einsum("oiab,niyxab->noyxab", u, v)
    y = np.einsum("ia,noyxab,jb->noyixj", at, mm, at)
    return y.reshape(n, f.shape[0], m * th, m * tw)[:, :, :h, :w]
