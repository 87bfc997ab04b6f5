"""Weight quantization error of the quantization strategies the paper compares
(Sec. V, the quantization-error figure and the discussion of channel-wise
versus tap-wise quantization): one scale per layer, per output channel, per
Winograd tap, or per (output channel, tap), with scales either free (fp32,
s = max|w| / 2^(n-1)) or rounded up to a power of two (Sec. III-B), in the
spatial domain (f) and in the Winograd domain (U = G f G^T).

Test infrastructure only: used by tests/ to check the paper's claims on the
synthetic layers that stand in for its networks.
"""
from fractions import Fraction

import numpy as np

from . import quant, tapwise

STRATEGIES = ("layer", "channel", "tap", "channel_tap")


def winograd_weights(f, m=4):
    """U = G f G^T in float64 [cout, cin, n, n] (from the exact plan arithmetic,
    rounded once to float64)."""
    spec = tapwise.SPECS[m]
    unum, p = tapwise.weight_transform_exact(f, spec)
    d2 = spec.den * spec.den
    scale = float(Fraction(2) ** p / d2)
    return np.vectorize(lambda v: float(v))(unum).astype(np.float64) * scale


def _group_absmax(w, strategy):
    """max |w| over each quantization group, broadcastable to w
    [cout, cin, k, k]: layer -> one value, channel -> per cout,
    tap -> per (a, b), channel_tap -> per (cout, a, b)."""
    a = np.abs(w)
    if strategy == "layer":
        return a.max(keepdims=True).reshape(1, 1, 1, 1)
    if strategy == "channel":
        return a.max(axis=(1, 2, 3), keepdims=True)
    if strategy == "tap":
        return a.max(axis=(0, 1), keepdims=True)
    if strategy == "channel_tap":
        return a.max(axis=1, keepdims=True)
    raise ValueError(strategy)


def quantize(w, strategy, pow2=True, bits=8):
    """Fake-quantized weights: per group s = max|w| / 2^(bits-1) (Eq. quant),
    s -> 2^ceil(log2 s) when pow2, q = clamp(R(w / s)), returned as q * s."""
    amax = _group_absmax(w, strategy)
    qmax = 2 ** (bits - 1)
    s = amax / qmax
    if pow2:
        # smallest e with amax <= 2^(bits-1) 2^e, exactly (cexp on each group)
        e = np.vectorize(lambda v: quant.cexp(Fraction(float(v)) * 128 / qmax) if v > 0 else 0)(amax)
        s = np.ldexp(1.0, e.astype(np.int64))
    s = np.where(s > 0, s, 1.0)
    q = np.clip(np.floor(w / s + 0.5), -qmax, qmax - 1)
    return q * s


def relative_error(w, wq):
    """||w - wq||_F / ||w||_F."""
    n = np.linalg.norm(w)
    return float(np.linalg.norm(w - wq) / n) if n > 0 else 0.0


def study(layers, m=4, bits=8):
    """Relative quantization error of every strategy on every layer:
    {(domain, strategy, pow2): [error per layer]} with domain 'spatial'
    (f; only layer and channel strategies apply) or 'winograd' (U)."""
    out = {}
    for f in layers:
        f = np.asarray(f, dtype=np.float32)
        u = winograd_weights(f, m)
        for pow2 in (True, False):
            for st in ("layer", "channel"):
                out.setdefault(("spatial", st, pow2), []).append(
                    relative_error(f.astype(np.float64), quantize(f.astype(np.float64), st, pow2, bits)))
            for st in STRATEGIES:
                out.setdefault(("winograd", st, pow2), []).append(relative_error(u, quantize(u, st, pow2, bits)))
    return out
