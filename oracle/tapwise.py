"""Tap-wise quantized integer Winograd F(4x4, 3x3) (Sec. III, Eq. winograd,
Eq. quant, the rearranged tap-wise scheme, and power-of-two scales of
Sec. III-B), plus the float64 Winograd algorithm it approximates.

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
"""
from fractions import Fraction

import numpy as np

from . import f4, quant

NTAP = 36
BT = f4.BT4_I          # 6x6
AT = f4.AT4_I          # 4x6
G24 = f4.G4_INT        # 6x3 integers, G = G24 / 24


# ---------------------------------------------------------------------------
# offline plan
# ---------------------------------------------------------------------------
def weight_transform_exact(f):
    """Exact U = G f G^T for fp32 weights f [cout, cin, 3, 3].

    Returns (unum, p): unum is an object array of Python ints with shape
    [cout, cin, 6, 6] and U = unum * 2^p / 576 exactly.
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
    g = np.array(G24, dtype=object)                   # 6x3
    unum = np.matmul(np.matmul(g, F), g.T)            # [cout, cin, 6, 6]
    return unum, p


def _u_abs_max_per_tap(unum, p):
    """max over (co, ci) of |U_t| for every tap, as exact Fractions."""
    out = []
    flat = unum.reshape(-1, NTAP)
    for t in range(NTAP):
        mx = max((abs(v) for v in flat[:, t]), default=0)
        out.append(Fraction(mx) * Fraction(2) ** p / 576)
    return out


def _quantize_unum(unum, p, e_g):
    """Uq = clamp(R(U / 2^e_G)) with U = unum * 2^p / 576, per tap."""
    cout, cin = unum.shape[:2]
    flat = unum.reshape(cout, cin, NTAP)
    uq = np.zeros((cout, cin, NTAP), dtype=np.int64)
    for t in range(NTAP):
        s = p - e_g[t]
        col = flat[:, :, t]
        if s >= 0:
            num = 2 * col * (1 << s) + 576
            den = 1152
        else:
            num = 2 * col + 576 * (1 << -s)
            den = 1152 * (1 << -s)
        q = num // den                                 # floor division
        uq[:, :, t] = np.clip(q.astype(np.int64) if q.dtype != object
                              else np.array([[int(v) for v in row] for row in q], dtype=np.int64),
                              quant.QMIN, quant.QMAX)
    return uq


def make_plan(f, e_b, e_g=None, bias=None, out_shift=0, relu=False):
    """The offline step: returns a dict with e_B, e_G, e, e_o, sh, Uq
    [36, cin, cout] (tap-major GEMM operand), bias [cout], out_shift, relu."""
    f = np.asarray(f, dtype=np.float32)
    cout, cin = f.shape[:2]
    e_b = [int(v) for v in e_b]
    assert len(e_b) == NTAP
    unum, p = weight_transform_exact(f)
    if e_g is None:
        e_g = [quant.cexp(a) for a in _u_abs_max_per_tap(unum, p)]
    else:
        e_g = [int(v) for v in e_g]
        assert len(e_g) == NTAP
    uq = _quantize_unum(unum, p, e_g)                 # [cout, cin, 36]
    e = [e_b[t] + e_g[t] for t in range(NTAP)]
    e_o = min(e)
    sh = [e[t] - e_o for t in range(NTAP)]
    if bias is None:
        bias = np.zeros(cout, dtype=np.int64)
    return dict(cin=cin, cout=cout, e_b=e_b, e_g=e_g, e=e, e_o=e_o, sh=sh,
                uq=np.ascontiguousarray(uq.transpose(2, 1, 0)),   # [36, cin, cout]
                bias=np.asarray(bias, dtype=np.int64).copy(),
                out_shift=int(out_shift), relu=bool(relu))


# ---------------------------------------------------------------------------
# online integer pipeline, batched formulation
# ---------------------------------------------------------------------------
def tile_grid(h, w):
    return -(-h // 4), -(-w // 4)


def input_tiles(x):
    """d[n, ci, ty, tx, r, c] = x[n, ci, 4ty + r - 1, 4tx + c - 1], zero
    outside the image."""
    x = np.asarray(x, dtype=np.int64)
    n, cin, h, w = x.shape
    th, tw = tile_grid(h, w)
    p = np.zeros((n, cin, 4 * th + 2, 4 * tw + 2), dtype=np.int64)
    p[:, :, 1:h + 1, 1:w + 1] = x
    d = np.zeros((n, cin, th, tw, 6, 6), dtype=np.int64)
    for r in range(6):
        for c in range(6):
            d[:, :, :, :, r, c] = p[:, :, r:r + 4 * th:4, c:c + 4 * tw:4]
    return d


def input_transform(d):
    """V = B^T d B on every tile (exact int64)."""
    return np.einsum("ar,...rc,bc->...ab", BT, d, BT)


def quantize_input_taps(v, e_b):
    """Vq[..., a, b] = clamp(R(V[..., a, b] / 2^e_B[6a+b]))."""
    vq = np.empty_like(v)
    for t in range(NTAP):
        a, b = divmod(t, 6)
        vq[..., a, b] = quant.clamp_int8(quant.shift_round_int(v[..., a, b], e_b[t]))
    return vq


def tap_major(vq):
    """[n, cin, th, tw, 6, 6] -> [36, T, cin] with tile index (n*th + ty)*tw + tx."""
    n, cin, th, tw = vq.shape[:4]
    return np.ascontiguousarray(vq.reshape(n, cin, th * tw, NTAP).transpose(3, 0, 2, 1)
                                .reshape(NTAP, n * th * tw, cin))


def tap_gemm(vq_tm, uq):
    """M[t] = Vq[t] @ Uq[t]: [36, T, cin] x [36, cin, cout] -> int64 [36, T, cout].
    Evaluated with float64 BLAS, exact because every partial sum is an
    integer of magnitude <= 2^14 * cin < 2^53."""
    cin = vq_tm.shape[2]
    assert cin < (1 << 38)
    m = np.matmul(vq_tm.astype(np.float64), uq.astype(np.float64))
    return m.astype(np.int64)


def output_transform(m, sh):
    """Y = A^T (M (.) 2^sh) A.  m [36, T, cout] -> Y [T, cout, 4, 4] (int64).
    The caller guarantees no int64 overflow (checked here)."""
    nt, cout = m.shape[1:]
    mm = np.empty_like(m)
    for t in range(NTAP):
        assert sh[t] < 40
        mm[t] = m[t] * (np.int64(1) << np.int64(sh[t]))
    assert np.abs(mm).max(initial=0) < (1 << 50)
    m6 = mm.reshape(6, 6, nt, cout).transpose(2, 3, 0, 1)        # [T, cout, 6, 6]
    return np.einsum("ia,...ab,jb->...ij", AT, m6, AT)


def assemble(yt, n, h, w):
    """[T, cout, 4, 4] tiles -> [n, cout, h, w], dropping out-of-image rows/cols."""
    th, tw = tile_grid(h, w)
    cout = yt.shape[1]
    y = yt.reshape(n, th, tw, cout, 4, 4).transpose(0, 3, 1, 4, 2, 5)
    return y.reshape(n, cout, 4 * th, 4 * tw)[:, :, :h, :w]


def prequant_output(x, plan):
    """z = Y + bias on in-image outputs, [n, cout, h, w] int64."""
    x = np.asarray(x)
    n, cin, h, w = x.shape
    assert cin == plan["cin"]
    v = input_transform(input_tiles(x))
    vq = quantize_input_taps(v, plan["e_b"])
    m = tap_gemm(tap_major(vq), plan["uq"])
    y = assemble(output_transform(m, plan["sh"]), n, h, w)
    return y + plan["bias"][None, :, None, None]


def requant(z, out_shift, relu):
    out = quant.clamp_int8(quant.shift_round_int(z, out_shift))
    if relu:
        out = np.maximum(out, 0)
    return out.astype(np.int8)


def conv_int8(x, plan):
    """The whole online path on int8 NCHW input: int8 NCHW output."""
    return requant(prequant_output(x, plan), plan["out_shift"], plan["relu"])


def input_taps_quantized(x, e_b):
    """Vq in tap-major layout [36, T, cin] (what the input-transform stage emits)."""
    return tap_major(quantize_input_taps(input_transform(input_tiles(x)), e_b))


# ---------------------------------------------------------------------------
# online integer pipeline, naive per-tile formulation (independent spelling)
# ---------------------------------------------------------------------------
def conv_int8_naive(x, plan):
    """Same definition, written as scalar loops over tiles, channels and taps
    with Python integers.  Only for tiny shapes."""
    x = np.asarray(x, dtype=np.int64)
    n, cin, h, w = x.shape
    cout = plan["cout"]
    th, tw = tile_grid(h, w)
    uq = plan["uq"]
    bt = f4.BT4
    at = f4.AT4
    out = np.zeros((n, cout, h, w), dtype=np.int8)

    def px(b, ci, r, c):
        return int(x[b, ci, r, c]) if 0 <= r < h and 0 <= c < w else 0

    for b in range(n):
        for ty in range(th):
            for tx in range(tw):
                vq = []                                   # vq[ci][t]
                for ci in range(cin):
                    d = [[px(b, ci, 4 * ty + r - 1, 4 * tx + c - 1) for c in range(6)]
                         for r in range(6)]
                    row = []
                    for t in range(NTAP):
                        a, bb = divmod(t, 6)
                        v = sum(bt[a][r] * d[r][c] * bt[bb][c]
                                for r in range(6) for c in range(6))
                        q = quant.clamp(quant.round_half_up(Fraction(v, 2 ** plan["e_b"][t])))
                        row.append(q)
                    vq.append(row)
                for co in range(cout):
                    msh = []
                    for t in range(NTAP):
                        acc = sum(vq[ci][t] * int(uq[t, ci, co]) for ci in range(cin))
                        msh.append(acc * 2 ** plan["sh"][t])
                    for i in range(4):
                        for j in range(4):
                            yy, xx = 4 * ty + i, 4 * tx + j
                            if yy >= h or xx >= w:
                                continue
                            val = sum(at[i][t // 6] * at[j][t % 6] * msh[t] for t in range(NTAP))
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


def input_tap_absmax(x):
    v = input_transform(input_tiles(x))
    return [int(np.abs(v[..., t // 6, t % 6]).max(initial=0)) for t in range(NTAP)]


def calibrate_input_exps(x):
    """e_B[t] = max(0, cexp(max over tiles and channels of |V_t|)), <= 15."""
    return [min(EB_MAX, max(0, quant.cexp(a))) for a in input_tap_absmax(x)]


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
      max_co max_ij sum_t |A^T[i,a] A^T[j,b]| 2^sh[t] 128 sum_ci |Uq[t,ci,co]|
      + max|bias| + (2^(out_shift-1) if out_shift > 0)."""
    uq = plan["uq"]
    s = np.abs(uq).sum(axis=1)                                 # [36, cout]
    best = 0
    for co in range(plan["cout"]):
        for i in range(4):
            for j in range(4):
                tot = 0
                for t in range(NTAP):
                    a, b = divmod(t, 6)
                    tot += abs(int(AT[i, a]) * int(AT[j, b])) * (1 << plan["sh"][t]) * 128 * int(s[t, co])
                best = max(best, tot)
    rnd = (1 << (plan["out_shift"] - 1)) if plan["out_shift"] > 0 else 0
    return best + int(np.abs(plan["bias"]).max(initial=0)) + rnd


def quantization_error_bound(x, f, plan, clamped_slack=False):
    """Per-output bound on |Y * 2^e_o - direct_fp64(x, f)| (before bias and
    requant): sum_t |A^T[i,a] A^T[j,b]| sum_ci (dB |U_t| + |V_t| dG + dB dG)
    with dB = 2^(e_B-1), dG = 2^(e_G-1) (2^e with ``clamped_slack`` to also
    cover the single +128 -> 127 saturation).  Returns [n, cout, h, w] float64."""
    x = np.asarray(x)
    n, cin, h, w = x.shape
    unum, p = weight_transform_exact(f)
    u_abs = np.abs(np.array([[[float(Fraction(int(v)) * Fraction(2) ** p / 576) for v in blk.ravel()]
                               for blk in row] for row in unum]))           # [cout, cin, 36]
    v = input_transform(input_tiles(x))                                      # [n,cin,th,tw,6,6]
    v_abs = np.abs(tap_major(v)).astype(np.float64)                          # [36, T, cin]
    k = 0 if clamped_slack else 1
    db = np.array([2.0 ** (plan["e_b"][t] - k) for t in range(NTAP)])
    dg = np.array([2.0 ** (plan["e_g"][t] - k) for t in range(NTAP)])
    ua = u_abs.transpose(2, 1, 0)                                            # [36, cin, cout]
    err = (db[:, None, None] * ua.sum(axis=1)[:, None, :]
           + dg[:, None, None] * v_abs.sum(axis=2)[:, :, None]
           + (db * dg)[:, None, None] * cin)                                # [36, T, cout]
    coef = np.abs(np.einsum("ia,jb->ijab", AT, AT)).reshape(4, 4, NTAP).astype(np.float64)
    bt = np.einsum("ijt,tkc->kcij", coef, err)                               # [T, cout, 4, 4]
    return assemble(bt, n, h, w)


# ---------------------------------------------------------------------------
# float64 Winograd F4 without quantization (Eq. winograd)
# ---------------------------------------------------------------------------
def conv_winograd_f64(x, f):
    x = np.asarray(x, dtype=np.float64)
    f = np.asarray(f, dtype=np.float64)
    n, cin, h, w = x.shape
    g = f4.G4_F
    bt = f4.BT4_I.astype(np.float64)
    at = f4.AT4_I.astype(np.float64)
    u = np.einsum("ar,oirc,bc->oiab", g, f, g)                    # [cout, cin, 6, 6]
    th, tw = tile_grid(h, w)
    p = np.zeros((n, cin, 4 * th + 2, 4 * tw + 2))
    p[:, :, 1:h + 1, 1:w + 1] = x
    d = np.zeros((n, cin, th, tw, 6, 6))
    for r in range(6):
        for c in range(6):
            d[:, :, :, :, r, c] = p[:, :, r:r + 4 * th:4, c:c + 4 * tw:4]
    v = np.einsum("ar,niyxrc,bc->niyxab", bt, d, bt)
    m = np.einsum("oiab,niyxab->noyxab", u, v)
    y = np.einsum("ia,noyxab,jb->noyixj", at, m, at)
    return y.reshape(n, f.shape[0], 4 * th, 4 * tw)[:, :, :h, :w]
