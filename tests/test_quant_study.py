"""The paper's weight-quantization comparison (Sec. V, quantization-error
figure; Sec. III, Challenge I) reproduced on the synthetic layers of C1-C5:
relative error of layer-, channel-, tap- and channel&tap-wise int8
quantization of the Winograd-domain weights U = G f G^T, with power-of-two
and free scales.  Claims checked:
  * F4 taps have very different dynamic ranges, so one scale for the whole
    Winograd-domain layer loses far more than it does in the spatial domain;
  * tap-wise quantization removes most of that loss (the paper: mean error
    2^-5.58 uniform -> 2^-6.78 tap-wise on ResNet-34) and beats channel-wise;
  * channel&tap-wise improves slightly further;
  * F2's taps are much closer in range (the problem is specific to F4);
  * power-of-two scales cost at most about one bit (error <= ~2x)."""
import numpy as np
import pytest

import workloads
from oracle import quant_study as qs


def _layers():
    out = []
    for name in ("C1", "C2", "C3", "C4", "C5"):
        _, ls = workloads.generate(name)
        out += [f for f, _, _ in ls]
    return out


@pytest.fixture(scope="module")
def res4():
    return qs.study(_layers(), m=4)


@pytest.fixture(scope="module")
def res2():
    return qs.study(_layers(), m=2)


def _mean(res, *key):
    return float(np.mean(res[key]))


def test_tapwise_beats_layerwise_and_channelwise_f4(res4):
    layer = _mean(res4, "winograd", "layer", True)
    chan = _mean(res4, "winograd", "channel", True)
    tap = _mean(res4, "winograd", "tap", True)
    both = _mean(res4, "winograd", "channel_tap", True)
    assert tap < layer / 2                  # the paper: 2.3x
    assert tap < chan / 2
    assert both <= tap
    # per layer, too
    for a, b in zip(res4[("winograd", "tap", True)], res4[("winograd", "layer", True)]):
        assert a < b


def test_f4_winograd_domain_is_harder_than_spatial(res4):
    assert _mean(res4, "winograd", "layer", True) > 3 * _mean(res4, "spatial", "layer", True)
    # with tap-wise scales the Winograd-domain error is back near the spatial one
    assert _mean(res4, "winograd", "tap", True) < 1.5 * _mean(res4, "spatial", "layer", True)


def test_f2_taps_have_similar_ranges(res2, res4):
    # layer-wise F2 in the Winograd domain is within 1.5x of spatial layer-wise,
    # and far better than layer-wise F4
    assert _mean(res2, "winograd", "layer", True) < 1.5 * _mean(res2, "spatial", "layer", True)
    assert _mean(res2, "winograd", "layer", True) < _mean(res4, "winograd", "layer", True) / 3


def test_power_of_two_scales_cost_at_most_about_one_bit(res4):
    for st in qs.STRATEGIES:
        p = _mean(res4, "winograd", st, True)
        f = _mean(res4, "winograd", st, False)
        assert f <= p <= 2.2 * f


def test_quantize_groups_and_pow2_rule():
    """The grouping and the scale rule on a hand-made tensor."""
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
