"""Weight quantization error of the grouping strategies the paper compares in
Sec. V-A ("Tap-wise vs. Channel-wise Quantization", the quantization-error
figure): one quantization group per layer, per output channel, per Winograd
tap, or per (output channel, tap), in the spatial domain (f) and in the
Winograd domain (U = G f G^T, mapped back to the spatial domain before the
error is measured).

The paper's procedure, as implemented here:
  * every group gets its own mean mu and standard deviation sigma, and the
    n-bit quantizer Quant_{mu,s}(x) = mu + s * clamp(R((x - mu) / s)) with
    the clamp to the signed n-bit range [-2^(n-1), 2^(n-1) - 1];
  * s = gamma * sigma / 2^(n-1), with gamma chosen per group to minimise the
    summed relative error sum_x |Quant_{mu,s}(x) - x| / |x|;
  * Winograd-domain weights are quantized as Quant(G f G^T) and brought back
    to the spatial domain with the Moore-Penrose inverse of G, computed from
    its singular value decomposition: f~ = G+ Quant(U) G+^T;
  * the reported figure is the distribution of the element-wise relative
    error |f~ - f| / |f| over all weights of all 3x3 layers, on a log2 scale,
    and its mean.

Readings where the paper is silent: sigma is the population standard deviation (divisor N);
R is round-half-up, as everywhere in this repository; gamma is the best of
the logarithmic grid 2^(k/16), k = -32..96 (gamma from 1/4 to 64), every
point evaluated, the smallest gamma winning a tie; weights equal to zero are left out of both the objective and
the error (their relative error is undefined); the "mean relative error"
is the mean of log2 |f~ - f| / |f| over the weights whose error is nonzero
(the mean of the plotted log2 distribution; an arithmetic mean of relative
errors diverges with weights near zero).

For comparison the module also evaluates the library's own scheme (Sec.
III-B): mu = 0 and power-of-two scales from the group's maximum magnitude,
s = 2^e with e the smallest exponent such that max |x| <= 2^(n-1) 2^e.

Test infrastructure only: used by tests/ to check the paper's claims on the
synthetic layers that stand in for its networks.
"""
from fractions import Fraction

import numpy as np

from . import f4, quant, tapwise

STRATEGIES = ("layer", "channel", "tap", "channel_tap")

GAMMA_STEPS = 16             # gamma grid 2^(k/16) ...
GAMMA_LOG2_MIN = -2          # ... from 1/4 ...
GAMMA_LOG2_MAX = 6           # ... to 64


# ---------------------------------------------------------------------------
# transforms
# ---------------------------------------------------------------------------
def transform_g(m=4):
    """G of F(m x m, 3 x 3) as float64 (Sec. II, the transform matrices)."""
    g = f4.G4 if m == 4 else f4.G2
    return np.array([[float(v) for v in row] for row in g], dtype=np.float64)


def pinv_svd(a):
    """Moore-Penrose inverse from the singular value decomposition a = W S V^T:
    a+ = V S+ W^T, where S+ inverts the singular values above the usual
    cut-off max(rows, cols) * eps * s_max and zeroes the rest."""
    a = np.asarray(a, dtype=np.float64)
    w, s, vt = np.linalg.svd(a, full_matrices=False)
    cut = max(a.shape) * np.finfo(np.float64).eps * (s.max() if s.size else 0.0)
    sinv = np.array([1.0 / v if v > cut else 0.0 for v in s])
    return (vt.T * sinv) @ w.T


def winograd_weights(f, m=4):
    """U = G f G^T in float64 [cout, cin, n, n] (from the exact plan arithmetic,
    rounded once to float64)."""
    spec = tapwise.SPECS[m]
    unum, p = tapwise.weight_transform_exact(f, spec)
    d2 = spec.den * spec.den
    scale = float(Fraction(2) ** p / d2)
    return np.vectorize(lambda v: float(v))(unum).astype(np.float64) * scale


def back_project(u, m=4):
    """Spatial weights from Winograd-domain ones: G+ u G+^T for every
    (cout, cin) of u [cout, cin, n, n]; returns [cout, cin, 3, 3]."""
    gp = pinv_svd(transform_g(m))                      # 3 x n
    return np.einsum("ia,ocab,jb->ocij", gp, u, gp)


# ---------------------------------------------------------------------------
# groups
# ---------------------------------------------------------------------------
def to_groups(w, strategy):
    """w [cout, cin, k, k] as a 2-D array [groups, members]: layer -> one group;
    channel -> one per output channel; tap -> one per (a, b) across all
    channels; channel_tap -> one per (cout, a, b) across input channels."""
    co, ci, k, _ = w.shape
    if strategy == "layer":
        return w.reshape(1, -1)
    if strategy == "channel":
        return w.reshape(co, -1)
    if strategy == "tap":
        return w.transpose(2, 3, 0, 1).reshape(k * k, co * ci)
    if strategy == "channel_tap":
        return w.transpose(0, 2, 3, 1).reshape(co * k * k, ci)
    raise ValueError(strategy)


def from_groups(g, shape, strategy):
    """Inverse of to_groups."""
    co, ci, k, _ = shape
    if strategy in ("layer", "channel"):
        return g.reshape(shape)
    if strategy == "tap":
        return g.reshape(k, k, co, ci).transpose(2, 3, 0, 1)
    if strategy == "channel_tap":
        return g.reshape(co, k, k, ci).transpose(0, 3, 1, 2)
    raise ValueError(strategy)


# ---------------------------------------------------------------------------
# the paper's quantizer and its scale search
# ---------------------------------------------------------------------------
def quant_mu_s(x, mu, s, bits=8):
    """Quant_{mu,s}(x) = mu + s * clamp(R((x - mu) / s), -2^(bits-1), 2^(bits-1) - 1)."""
    qmax = 2 ** (bits - 1)
    return mu + s * np.clip(np.floor((x - mu) / s + 0.5), -qmax, qmax - 1)


def group_stats(x):
    """Per-group mean and population standard deviation of x [groups, members]."""
    mu = x.mean(axis=1, keepdims=True)
    sigma = np.sqrt(((x - mu) ** 2).mean(axis=1, keepdims=True))
    return mu, sigma


def gamma_objective(x, gammas, bits=8):
    """sum over each group's nonzero members of |Quant_{mu,s}(x) - x| / |x|
    with s = gamma sigma / 2^(bits-1): array [len(gammas), groups]."""
    mu, sigma = group_stats(x)
    sigma = np.where(sigma > 0, sigma, 1.0)
    nz = x != 0
    inv = np.where(nz, 1.0 / np.where(nz, np.abs(x), 1.0), 0.0)
    out = np.empty((len(gammas), x.shape[0]))
    for i, g in enumerate(gammas):
        s = g * sigma / 2 ** (bits - 1)
        out[i] = (np.abs(quant_mu_s(x, mu, s, bits) - x) * inv).sum(axis=1)
    return out


def gamma_grid():
    """The candidate gammas: 2^(k/16) from 2^-2 to 2^6."""
    k = np.arange(GAMMA_LOG2_MIN * GAMMA_STEPS, GAMMA_LOG2_MAX * GAMMA_STEPS + 1)
    return 2.0 ** (k / GAMMA_STEPS)


def gamma_hat(x, bits=8):
    """Per group, the grid gamma with the smallest gamma_objective (the
    smallest such gamma on ties).  The objective is far from unimodal in
    gamma -- a few members near zero dominate it -- so every grid point is
    evaluated."""
    grid = gamma_grid()
    return grid[np.argmin(gamma_objective(x, grid, bits), axis=0)]


def paper_quantize(w, strategy, bits=8):
    """Weights quantized by the paper's procedure with one (mu, sigma, gamma)
    per group; returns (w quantized, gamma per group)."""
    x = to_groups(np.asarray(w, dtype=np.float64), strategy)
    g = gamma_hat(x, bits)
    mu, sigma = group_stats(x)
    s = g[:, None] * np.where(sigma > 0, sigma, 1.0) / 2 ** (bits - 1)
    return from_groups(quant_mu_s(x, mu, s, bits), w.shape, strategy), g


# ---------------------------------------------------------------------------
# the library's scheme: mu = 0, power-of-two (or free) max-abs scales
# ---------------------------------------------------------------------------
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
    """Fake-quantized weights of the library's scheme: per group s = max|w| /
    2^(bits-1) (Eq. quant), s -> 2^ceil(log2 s) when pow2, q = clamp(R(w / s)),
    returned as q * s."""
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


# ---------------------------------------------------------------------------
# the error measure and the study
# ---------------------------------------------------------------------------
def log2_relative_errors(f, fq):
    """log2 |fq - f| / |f| for every weight with f != 0 and a nonzero error,
    and the number of nonzero weights reproduced exactly."""
    f = np.asarray(f, dtype=np.float64).ravel()
    fq = np.asarray(fq, dtype=np.float64).ravel()
    nz = f != 0
    r = np.abs(fq[nz] - f[nz]) / np.abs(f[nz])
    return np.log2(r[r > 0]), int((r == 0).sum())


def study(layers, m=4, bits=8):
    """Every layer through every strategy: {(domain, strategy, scheme): array of
    log2 relative errors, all layers pooled}.  domain 'spatial' quantizes f
    (layer and channel groups), 'winograd' quantizes U = G f G^T and back-
    projects; scheme 'paper' is the (mu, sigma, gamma) procedure, 'pow2' the
    library's max-abs power-of-two scales."""
    out = {}
    for f in layers:
        f64 = np.asarray(f, dtype=np.float32).astype(np.float64)
        u = winograd_weights(np.asarray(f, dtype=np.float32), m)
        for st in ("layer", "channel"):
            out.setdefault(("spatial", st, "paper"), []).append(
                log2_relative_errors(f64, paper_quantize(f64, st, bits)[0])[0])
            out.setdefault(("spatial", st, "pow2"), []).append(
                log2_relative_errors(f64, quantize(f64, st, True, bits))[0])
        for st in STRATEGIES:
            out.setdefault(("winograd", st, "paper"), []).append(
                log2_relative_errors(f64, back_project(paper_quantize(u, st, bits)[0], m))[0])
            out.setdefault(("winograd", st, "pow2"), []).append(
                log2_relative_errors(f64, back_project(quantize(u, st, True, bits), m))[0])
    return {k: np.concatenate(v) for k, v in out.items()}


def mean_log2(res, *key):
    """The study's headline figure for one row: mean log2 relative error."""
    return float(np.mean(res[key]))
