"""The paper's weight-quantization comparison (Sec. V-A, "Tap-wise vs.
Channel-wise Quantization", and the quantization-error figure) on synthetic
3x3 layers: per-group mean, standard deviation and searched scale factor,
Winograd-domain weights back-projected through the SVD pseudo-inverse of G,
and the mean log2 relative error of the spatial weights.

The first half pins oracle/quant_study.py to things other than itself
(exact rational inverses, closed forms, brute force in exact arithmetic,
planted mistakes); the second half checks the paper's claims on the layers
of C1-C3 and on the same layers with per-channel scales."""
from fractions import Fraction as Fr

import numpy as np
import pytest

import workloads
from oracle import f4
from oracle import quant_study as qs


# ---------------------------------------------------------------------------
# pins
# ---------------------------------------------------------------------------
def _exact_left_inverse(g):
    """(G^T G)^-1 G^T in exact rationals (G has full column rank 3)."""
    n = len(g)
    gtg = [[sum(g[k][i] * g[k][j] for k in range(n)) for j in range(3)] for i in range(3)]
    # Gauss-Jordan on [G^T G | G^T]
    aug = [list(gtg[i]) + [g[k][i] for k in range(n)] for i in range(3)]
    for c in range(3):
        p = next(r for r in range(c, 3) if aug[r][c] != 0)
        aug[c], aug[p] = aug[p], aug[c]
        piv = aug[c][c]
        aug[c] = [v / piv for v in aug[c]]
        for r in range(3):
            if r != c and aug[r][c] != 0:
                fac = aug[r][c]
                aug[r] = [a - fac * b for a, b in zip(aug[r], aug[c])]
    return [row[3:] for row in aug]


@pytest.mark.parametrize("m,g", [(4, f4.G4), (2, f4.G2)])
def test_pinv_equals_the_exact_left_inverse(m, g):
    """G is 6x3 (F4) or 4x3 (F2) with full column rank, so its Moore-Penrose
    inverse is the left inverse (G^T G)^-1 G^T, here in exact rationals."""
    exact = np.array([[float(v) for v in row] for row in _exact_left_inverse(g)])
    got = qs.pinv_svd(qs.transform_g(m))
    assert got.shape == (3, len(g))
    assert np.allclose(got, exact, rtol=1e-12, atol=1e-13)
    assert np.allclose(got @ qs.transform_g(m), np.eye(3), atol=1e-13)


def test_pinv_of_a_rank_deficient_matrix():
    """A rank-one matrix a = u v^T has a+ = a^T / ||a||_F^2; the four Penrose
    conditions hold."""
    a = np.outer([1.0, -2.0, 0.5], [3.0, 1.0, -1.0, 2.0])
    p = qs.pinv_svd(a)
    assert np.allclose(p, a.T / (a * a).sum(), atol=1e-14)
    assert np.allclose(a @ p @ a, a, atol=1e-12)
    assert np.allclose(p @ a @ p, p, atol=1e-14)
    assert np.allclose((a @ p).T, a @ p, atol=1e-14)
    assert np.allclose((p @ a).T, p @ a, atol=1e-14)


@pytest.mark.parametrize("m", [4, 2])
def test_back_projection_inverts_the_weight_transform(m):
    """G+ (G f G^T) G+^T = f for every (cout, cin); f is not symmetric, so a
    transposed operand would show."""
    f = np.random.default_rng(11).standard_normal((3, 2, 3, 3)).astype(np.float32)
    u = qs.winograd_weights(f, m)
    assert np.allclose(qs.back_project(u, m), f.astype(np.float64), rtol=0, atol=1e-12)


def test_back_projection_catches_a_planted_transpose(monkeypatch):
    """Planted mistake: G^T in place of G+ (a plausible slip) no longer
    inverts the transform, so the test above would fail."""
    f = np.random.default_rng(12).standard_normal((2, 2, 3, 3)).astype(np.float32)
    u = qs.winograd_weights(f, 4)
    monkeypatch.setattr(qs, "pinv_svd", lambda a: np.asarray(a).T)
    assert not np.allclose(qs.back_project(u, 4), f.astype(np.float64), atol=1e-3)


def _two_point_group(n=40, mu=7.5, d=0.75):
    """n members, half mu - d and half mu + d (dyadic values: every step below
    is exact)."""
    x = np.full((1, n), mu)
    x[0, : n // 2] -= d
    x[0, n // 2:] += d
    return x


def test_two_point_group_closed_form():
    """Members mu0 +- d: the group's mean is mu0 and its population standard
    deviation d, so s = gamma d / 128 puts both members exactly on the grid
    whenever 128 / gamma is an integer no larger than 127; the smallest grid
    gamma with that property is 2 (2^(k/16) for k < 16 gives no integer), and
    it reproduces the group exactly."""
    x = _two_point_group()
    g = qs.gamma_hat(x)
    assert g[0] == 2.0
    q, gam = qs.paper_quantize(x.reshape(1, 1, 8, 5), "layer")
    assert gam[0] == 2.0 and np.array_equal(q.reshape(1, -1), x)
    assert qs.gamma_objective(x, [2.0])[0, 0] == 0.0
    # a quarter of the way: gamma 4 puts the members at +-32 steps, also exact
    assert qs.gamma_objective(x, [4.0])[0, 0] == 0.0
    # gamma 1: 128 steps clamps to 127, so the upper member is off by d / 128
    assert qs.gamma_objective(x, [1.0])[0, 0] == pytest.approx(20 * (0.75 / 128) / 8.25, rel=1e-12)


@pytest.mark.parametrize("mistake", ["sample_std", "two_to_the_n", "no_mean"])
def test_two_point_group_catches_planted_mistakes(monkeypatch, mistake):
    """Planted mistakes in the quantizer: the sample standard deviation
    (divisor N - 1), 2^n in place of 2^(n-1), or a quantizer without the
    group mean each move the closed-form optimum away from gamma = 2."""
    x = _two_point_group()
    if mistake == "sample_std":
        def stats(v):
            mu = v.mean(axis=1, keepdims=True)
            return mu, np.sqrt(((v - mu) ** 2).sum(axis=1, keepdims=True) / (v.shape[1] - 1))
        monkeypatch.setattr(qs, "group_stats", stats)
    elif mistake == "two_to_the_n":
        real = qs.quant_mu_s
        monkeypatch.setattr(qs, "quant_mu_s", lambda v, mu, s, bits=8: real(v, mu, s / 2, bits))
    else:
        real = qs.quant_mu_s
        monkeypatch.setattr(qs, "quant_mu_s", lambda v, mu, s, bits=8: real(v, 0 * mu, s, bits))
    g = qs.gamma_hat(x)
    assert g[0] != 2.0 or qs.gamma_objective(x, [2.0])[0, 0] != 0.0


def _exact_objective(vals, gamma, bits=8):
    """sum |Quant(x) - x| / |x| in exact rationals for one group, gamma a
    float64 grid point (so a dyadic rational); sigma enters as the exact
    square root's float64 value, as it does in the vectorized code."""
    xs = [Fr(float(v)) for v in vals]
    n = len(xs)
    mu = sum(xs) / n
    var = sum((v - mu) ** 2 for v in xs) / n
    sigma = Fr(float(np.sqrt(float(var))))
    s = Fr(float(gamma)) * sigma / 2 ** (bits - 1)
    qmax = 2 ** (bits - 1)
    tot = Fr(0)
    for v in xs:
        if v == 0:
            continue
        k = (v - mu) / s + Fr(1, 2)
        k = min(max(k.numerator // k.denominator, -qmax), qmax - 1)
        tot += abs(mu + s * k - v) / abs(v)
    return tot


def test_gamma_search_against_exact_brute_force():
    """Tiny groups: the vectorized objective agrees with an exact-rational
    evaluation at every grid point, and gamma_hat is the first grid point
    where the exact objective is smallest (up to float64 ties)."""
    rng = np.random.default_rng(21)
    grid = qs.gamma_grid()
    groups = [rng.standard_normal(9), rng.laplace(size=7) * 0.3 + 0.1, np.array([0.0, 1.0, -2.0, 0.25, 3.5])]
    for vals in groups:
        x = vals.reshape(1, -1)
        vec = qs.gamma_objective(x, grid)[:, 0]
        exact = np.array([float(_exact_objective(vals, g)) for g in grid])
        assert np.allclose(vec, exact, rtol=1e-9, atol=1e-12)
        best = exact.min()
        g = qs.gamma_hat(x)[0]
        assert float(_exact_objective(vals, g)) <= best * (1 + 1e-9) + 1e-12
        first = grid[np.nonzero(exact <= best * (1 + 1e-9) + 1e-12)[0][0]]
        assert g == first


def test_mean_log2_error_closed_form_for_gaussian_weights():
    """For Gaussian weights and a fixed gamma = 4 (clipping ~1e-4 of them),
    the rounding error is uniform on [0, s/2] and independent of |f|, so
    E[log2 |e| / |f|] = log2(s / 2) - 1/ln 2 - E[log2 |f|] with
    E[log2 |Z|] = -(Euler's gamma + ln 2) / (2 ln 2) for Z ~ N(0, 1):
    log2(4 / 256) - 1/ln 2 + (0.5772... + ln 2) / (2 ln 2) = -6.526."""
    x = np.random.default_rng(31).standard_normal((1, 1 << 20)) * 0.03
    mu, sigma = qs.group_stats(x)
    q = qs.quant_mu_s(x, mu, 4 * sigma / 128)
    errs, exact = qs.log2_relative_errors(x, q)
    want = np.log2(4 / 256) - 1 / np.log(2) + (np.euler_gamma + np.log(2)) / (2 * np.log(2))
    assert abs(errs.mean() - want) < 0.01
    assert exact < 50


def test_log2_relative_errors_by_hand():
    f = np.array([1.0, 2.0, -4.0, 0.0])
    fq = np.array([1.5, 2.0, -3.5, 0.1])
    errs, exact = qs.log2_relative_errors(f, fq)
    assert sorted(errs.tolist()) == [-3.0, -1.0] and exact == 1      # 0.5, 0, 0.125; f = 0 left out


@pytest.mark.parametrize("strategy", qs.STRATEGIES)
def test_groups_round_trip_and_membership(strategy):
    w = np.arange(2 * 3 * 6 * 6, dtype=np.float64).reshape(2, 3, 6, 6)
    g = qs.to_groups(w, strategy)
    assert np.array_equal(qs.from_groups(g, w.shape, strategy), w)
    want = {"layer": [w.ravel()],
            "channel": [w[c].ravel() for c in range(2)],
            "tap": [w[:, :, a, b].ravel() for a in range(6) for b in range(6)],
            "channel_tap": [w[c, :, a, b] for c in range(2) for a in range(6) for b in range(6)]}[strategy]
    assert len(g) == len(want)
    for row, ref in zip(g, want):
        assert sorted(row.tolist()) == sorted(ref.tolist())


def test_quantize_groups_and_pow2_rule():
    """The library's scheme (mu = 0, max-abs power-of-two scales) on a
    hand-made tensor."""
    w = np.zeros((2, 1, 2, 2))
    w[0, 0] = [[1.0, -0.5], [0.25, 0.0]]
    w[1, 0] = [[8.0, 0.0], [0.0, -3.0]]
    # per channel, pow2: channel 0 max 1 -> s = 2^-7; channel 1 max 8 -> s = 2^-4;
    # each positive maximum sits at exactly 128 steps and clamps to 127
    q = qs.quantize(w, "channel", pow2=True)
    want = w.copy()
    want[0, 0, 0, 0] = 127 * 2.0 ** -7
    want[1, 0, 0, 0] = 127 * 2.0 ** -4
    assert np.array_equal(q, want)
    # layer-wise: s = 8/128 = 2^-4 for all; 1.0, -0.5, 0.25 are multiples of it
    want = w.copy()
    want[1, 0, 0, 0] = 127 * 2.0 ** -4
    assert np.array_equal(qs.quantize(w, "layer", pow2=True), want)
    # tap-wise groups (a, b) span all channels: tap (0,0) holds 1 and 8 -> s = 2^-4,
    # so 1.0 is exact; tap (1,0) holds only 0.25 -> s = 2^-9 and 0.25 saturates;
    # tap (1,1) max 3 -> s = 2^-5 (3 <= 128 * 2^-5 = 4), -3 is exact
    qt = qs.quantize(w, "tap", pow2=True)
    assert qt[0, 0, 0, 0] == 1.0 and qt[0, 0, 1, 0] == 127 * 2.0 ** -9
    assert qt[1, 0, 1, 1] == -3.0
    # channel&tap: each (cout, a, b) is its own group, so every nonzero positive
    # value is a group maximum and saturates; negative ones are exact
    qct = qs.quantize(w, "channel_tap", pow2=True)
    assert qct[0, 0, 0, 1] == -0.5 and qct[1, 0, 0, 0] == 8.0 * 127 / 128
    # a value that is not a multiple of the step rounds half up
    w2 = np.array([[[[1.0, 3 * 2.0 ** -8]]]])          # s = 2^-7 -> 1.5 steps -> 2 steps
    assert qs.quantize(w2, "layer", pow2=True)[0, 0, 0, 1] == 2 * 2.0 ** -7
    # the group's extreme values: -max is representable, +max saturates
    w3 = np.array([[[[128.0, -128.0]]]])
    q3 = qs.quantize(w3, "layer", pow2=True)
    assert q3[0, 0, 0, 0] == 127.0 and q3[0, 0, 0, 1] == -128.0


def test_winograd_weights_corner_taps():
    """The corner rows of G are (1/4, 0, 0) and (0, 0, 1) for F4 and
    (1, 0, 0), (0, 0, 1) for F2 (Sec. II, the transform matrices), so the
    corner taps of U are single weights; F2's second row of G is
    (1, 1, 1) / 2, so its tap (1, 1) is the kernel's sum over 4."""
    rng = np.random.default_rng(5)
    f = rng.standard_normal((3, 2, 3, 3)).astype(np.float32)
    u4 = qs.winograd_weights(f, 4)
    assert np.allclose(u4[:, :, 0, 0], f[:, :, 0, 0] / 16, rtol=1e-12, atol=0)
    assert np.allclose(u4[:, :, 5, 5], f[:, :, 2, 2], rtol=1e-12, atol=0)
    assert np.allclose(u4[:, :, 0, 5], f[:, :, 0, 2] / 4, rtol=1e-12, atol=0)
    u2 = qs.winograd_weights(f, 2)
    assert np.allclose(u2[:, :, 0, 0], f[:, :, 0, 0], rtol=1e-12, atol=0)
    assert np.allclose(u2[:, :, 3, 3], f[:, :, 2, 2], rtol=1e-12, atol=0)
    assert np.allclose(u2[:, :, 1, 1], f.astype(np.float64).sum(axis=(2, 3)) / 4, rtol=1e-12, atol=1e-15)


# ---------------------------------------------------------------------------
# the paper's claims on synthetic layers
# ---------------------------------------------------------------------------
def _layers(scaled):
    """The first four synthetic layers (C1, C2, the first two of C3); with
    scaled, each output channel multiplied by a log-normal factor."""
    out = []
    for name in ("C1", "C2", "C3"):
        _, ls = workloads.generate(name)
        out += [f for f, _, _ in ls]
    out = out[:4]
    if scaled:
        out = [workloads.channel_scaled(f, 100 + i) for i, f in enumerate(out)]
    return out


@pytest.fixture(scope="module")
def res4():
    return {sc: qs.study(_layers(sc), m=4) for sc in (False, True)}


@pytest.fixture(scope="module")
def res2():
    return qs.study(_layers(False), m=2)


def _m(res, *key):
    return qs.mean_log2(res, *key)


@pytest.mark.parametrize("scaled", [False, True])
def test_tapwise_beats_layerwise_and_channelwise_in_the_winograd_domain(res4, scaled):
    """The paper: uniform 2^-5.58 -> tap-wise 2^-6.78 (2.3x), channel-wise
    barely moving (2^-5.62), channel & tap a further 1.06x."""
    r = res4[scaled]
    layer, chan = _m(r, "winograd", "layer", "paper"), _m(r, "winograd", "channel", "paper")
    tap, both = _m(r, "winograd", "tap", "paper"), _m(r, "winograd", "channel_tap", "paper")
    assert tap < layer - 1.0
    assert tap < chan - 1.0
    assert chan > layer - 0.3            # channel-wise gains little (here it loses)
    assert both < tap


@pytest.mark.parametrize("scaled", [False, True])
def test_f4_winograd_domain_is_harder_than_spatial(res4, scaled):
    """One scale for F4's Winograd-domain weights costs more than one scale
    for the spatial ones (the paper: 2^-5.58 against 2^-6.01)."""
    r = res4[scaled]
    assert _m(r, "winograd", "layer", "paper") > _m(r, "spatial", "layer", "paper") + 0.3


def test_channelwise_helps_in_the_spatial_domain_only_when_channels_differ(res4):
    """The paper: 2^-6.01 -> 2^-6.72 (1.7x) spatially, on trained weights.
    Output channels with different scales reproduce the gain; i.i.d. draws,
    whose channels share one distribution, do not."""
    sc = res4[True]
    assert _m(sc, "spatial", "channel", "paper") < _m(sc, "spatial", "layer", "paper") - 0.3
    iid = res4[False]
    assert abs(_m(iid, "spatial", "channel", "paper") - _m(iid, "spatial", "layer", "paper")) < 0.1


def test_f2_taps_have_similar_ranges(res2, res4):
    """F2's transform barely spreads the taps, so one Winograd-domain scale
    stays close to the spatial one; F4's does not (Sec. II, Challenge I)."""
    assert _m(res2, "winograd", "layer", "paper") < _m(res2, "spatial", "layer", "paper") + 0.5
    assert _m(res2, "winograd", "layer", "paper") < _m(res4[False], "winograd", "layer", "paper") - 1.5


@pytest.mark.parametrize("scaled", [False, True])
def test_library_scheme_keeps_most_of_the_tapwise_gain(res4, scaled):
    """The kernels' scheme (mu = 0, power-of-two max-abs scales per tap,
    Sec. III-B) is within about one bit of the paper's searched tap-wise
    scales and still well ahead of any one-scale Winograd quantization."""
    r = res4[scaled]
    p2 = _m(r, "winograd", "tap", "pow2")
    assert p2 < _m(r, "winograd", "tap", "paper") + 1.5
    assert p2 < _m(r, "winograd", "layer", "paper") - 0.5
    assert p2 < _m(r, "winograd", "layer", "pow2") - 1.5
