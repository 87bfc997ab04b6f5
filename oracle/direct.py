"""Direct 3x3 convolution, stride 1, padding 1 (the "standard algorithm" the
paper compares against, Sec. I and Sec. III last paragraph).

y[n, co, h, w] = sum_{ci, r, c} x[n, ci, h + r - 1, w + c - 1] * f[co, ci, r, c]
with x taken as zero outside the image (cross-correlation, NCHW).

Three independent spellings:
  * conv_f64        float64, one shifted slice per kernel position;
  * conv_int        exact int64 accumulation, one shifted slice per position;
  * conv_bruteforce pure Python loops over every index, for tiny inputs.
plus the int8 direct convolution with power-of-two requantization that the
library's direct kernel must match bit for bit.
"""
import numpy as np

from . import quant


def _padded(x, dtype):
    n, c, h, w = x.shape
    p = np.zeros((n, c, h + 2, w + 2), dtype=dtype)
    p[:, :, 1:h + 1, 1:w + 1] = x
    return p


def conv_f64(x, f):
    x = np.asarray(x, dtype=np.float64)
    f = np.asarray(f, dtype=np.float64)
    n, cin, h, w = x.shape
    cout = f.shape[0]
    assert f.shape == (cout, cin, 3, 3)
    p = _padded(x, np.float64)
    y = np.zeros((n, cout, h, w), dtype=np.float64)
    for r in range(3):
        for c in range(3):
            win = p[:, :, r:r + h, c:c + w]            # [n, cin, h, w]
            y += np.einsum("nihw,oi->nohw", win, f[:, :, r, c])
    return y


def conv_int(x, f):
    """Exact integer accumulation; returns int64 [n, cout, h, w]."""
    x = np.asarray(x, dtype=np.int64)
    f = np.asarray(f, dtype=np.int64)
    n, cin, h, w = x.shape
    cout = f.shape[0]
    assert f.shape == (cout, cin, 3, 3)
    p = _padded(x, np.int64)
    y = np.zeros((n, cout, h, w), dtype=np.int64)
    for r in range(3):
        for c in range(3):
            win = p[:, :, r:r + h, c:c + w].transpose(0, 2, 3, 1).reshape(-1, cin)
            # float64 BLAS is exact here: every partial sum is an integer
            # below 2^53 (|x|,|f| <= 128 and cin <= 2^30).
            prod = win.astype(np.float64) @ f[:, :, r, c].T.astype(np.float64)
            y += prod.astype(np.int64).reshape(n, h, w, cout).transpose(0, 3, 1, 2)
    return y


def conv_bruteforce(x, f):
    """Pure Python loops; returns a nested-list-free numpy object array so
    exact rationals (Fractions) pass through unchanged."""
    n, cin, h, w = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    cout = len(f)
    y = np.empty((n, cout, h, w), dtype=object)
    for b in range(n):
        for co in range(cout):
            for i in range(h):
                for j in range(w):
                    acc = 0
                    for ci in range(cin):
                        for r in range(3):
                            for c in range(3):
                                hh, ww = i + r - 1, j + c - 1
                                if 0 <= hh < h and 0 <= ww < w:
                                    acc += x[b][ci][hh][ww] * f[co][ci][r][c]
                    y[b, co, i, j] = acc
    return y


def requant(z, out_shift, relu):
    """out = clamp(R(z / 2^out_shift), -128, 127), then max(out, 0) if relu."""
    out = quant.clamp_int8(quant.shift_round_int(z, out_shift))
    if relu:
        out = np.maximum(out, 0)
    return out.astype(np.int8)


def conv_int8(x, w_int8, bias, out_shift, relu):
    """Direct int8 convolution: int8 x and weights, int32 bias in accumulator
    units, power-of-two requantization.  Returns int8 NCHW."""
    z = conv_int(x, w_int8)
    if bias is not None:
        z = z + np.asarray(bias, dtype=np.int64)[None, :, None, None]
    return requant(z, out_shift, relu)


def quantize_weights_pow2(f):
    """Spatial int8 weights for the direct baseline: one power-of-two scale
    per layer from the max-abs weight, same R / clamp rule as the method.
    Returns (int8 weights, exponent e) with f ~ w * 2^e."""
    from fractions import Fraction
    f = np.asarray(f, dtype=np.float32)
    amax = max((Fraction(float(v)) for v in np.abs(f).ravel()), default=Fraction(0))
    e = quant.cexp(amax)
    flat = [quant.quantize_exact(Fraction(float(v)), e) for v in f.ravel()]
    return np.array(flat, dtype=np.int8).reshape(f.shape), e
