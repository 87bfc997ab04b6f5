"""Seeded synthetic workloads for the 3x3 convolution layers.

This module only draws inputs; it holds none of the method's arithmetic and
is shared by the tests, the benchmark and the smoke check.  Every draw uses
numpy's PCG64 generator (``default_rng(seed)``) in a fixed order per layer:
activations, then weights (then the outlier mask), then bias.  Activations
are drawn in NCHW order; NHWC callers transpose the same values.

Shapes stand in for the paper's workloads (Sec. V): its 63-layer synthetic
3x3 suite and the 3x3 layers of ResNet, UNet and detection networks, whose
tensors and weights are not available.  Distributions:
  C1 smoke       N=1, 16->16, 32x32: |N(0,1)|*20 rounded, clipped to 127;
                 weights N(0, 0.1); bias U[-64, 64]; out_shift 8
  C2 resnet-s1   N=8, 64->64, 56x56: 50% zeros, else |N(0,1)|*24; He-normal
  C3 resnet-4    N=8, four chained layers (64->128@56, 128->128@28,
                 128->256@28, 256->256@14); first input as C2; He-normal
  C4 unet-hr     N=1, 128->128, 256x512: 60% zeros, else |Laplace(0,1)|*16
  C5 det-neck    N=4, 256->256, 160x160: 50% zeros, else |N(0,1)|*24;
                 He-normal with 1% of entries scaled by 8; bias U[-256, 256]
"""
from dataclasses import dataclass, field

import numpy as np


@dataclass
class LayerSpec:
    cin: int
    cout: int
    h: int
    w: int
    bias_range: int = 64
    weights: str = "he"          # "he" or "normal0.1"
    outliers: float = 0.0        # fraction of weight entries scaled by 8
    relu: bool = False
    out_shift: int | None = None  # None = calibrated


@dataclass
class Workload:
    name: str
    n: int
    layers: list
    act: str                      # activation recipe of the first input
    zero_frac: float = 0.0
    seed: int = 0
    desc: str = ""
    chained: bool = False


WORKLOADS = {
    "C1": Workload("C1", 1, [LayerSpec(16, 16, 32, 32, weights="normal0.1", out_shift=8)],
                   act="halfnormal20", desc="single layer, N=1, 16->16, 32x32, NCHW"),
    "C2": Workload("C2", 8, [LayerSpec(64, 64, 56, 56)], act="halfnormal24", zero_frac=0.5,
                   desc="ResNet stage-1 3x3 layer, N=8, 64->64, 56x56"),
    "C3": Workload("C3", 8, [LayerSpec(64, 128, 56, 56, relu=True),
                             LayerSpec(128, 128, 28, 28, relu=True),
                             LayerSpec(128, 256, 28, 28, relu=True),
                             LayerSpec(256, 256, 14, 14, relu=True)],
                   act="halfnormal24", zero_frac=0.5, chained=True,
                   desc="four chained 3x3 layers, N=8"),
    "C4": Workload("C4", 1, [LayerSpec(128, 128, 256, 512)], act="laplace16", zero_frac=0.6,
                   desc="segmentation-backbone layer, N=1, 128->128, 256x512"),
    "C5": Workload("C5", 4, [LayerSpec(256, 256, 160, 160, bias_range=256, outliers=0.01)],
                   act="halfnormal24", zero_frac=0.5,
                   desc="detection-neck layer, N=4, 256->256, 160x160"),
}


def draw_activations(rng, shape, recipe, zero_frac):
    """int8 NCHW activations, non-negative (ReLU-like)."""
    zero = rng.random(shape) < zero_frac if zero_frac > 0 else None
    if recipe == "halfnormal20":
        v = np.abs(rng.standard_normal(shape)) * 20
    elif recipe == "halfnormal24":
        v = np.abs(rng.standard_normal(shape)) * 24
    elif recipe == "laplace16":
        v = np.abs(rng.laplace(0.0, 1.0, shape)) * 16
    elif recipe == "int8full":
        return rng.integers(-128, 128, shape).astype(np.int8)
    else:
        raise ValueError(recipe)
    a = np.clip(np.round(v), 0, 127)
    if zero is not None:
        a[zero] = 0
    return a.astype(np.int8)


def draw_weights(rng, spec):
    shape = (spec.cout, spec.cin, 3, 3)
    if spec.weights == "normal0.1":
        f = rng.normal(0.0, 0.1, shape)
    else:
        f = rng.normal(0.0, np.sqrt(2.0 / (9 * spec.cin)), shape)
    if spec.outliers > 0:
        f = np.where(rng.random(shape) < spec.outliers, f * 8, f)
    return f.astype(np.float32)


def channel_scaled(f, seed, sigma=0.5):
    """The weights f [cout, cin, 3, 3] with each output channel multiplied by
    its own log-normal factor exp(N(0, sigma^2)), drawn from default_rng(seed)
    in channel order.  Trained networks' output channels differ in scale, the
    property channel-wise quantization exploits; i.i.d. draws lack it."""
    rng = np.random.default_rng(seed)
    k = np.exp(rng.normal(0.0, sigma, f.shape[0]))
    return (f.astype(np.float64) * k[:, None, None, None]).astype(np.float32)


def draw_bias(rng, spec):
    return rng.integers(-spec.bias_range, spec.bias_range + 1, spec.cout).astype(np.int32)


def generate(name, n=None, seed=None):
    """Returns (x, layers): x int8 NCHW [n, cin, h, w] for the first layer and
    a list of (weights fp32 [cout, cin, 3, 3], bias int32 [cout], spec)."""
    wl = WORKLOADS[name]
    n = wl.n if n is None else n
    rng = np.random.default_rng(wl.seed if seed is None else seed)
    s0 = wl.layers[0]
    x = draw_activations(rng, (n, s0.cin, s0.h, s0.w), wl.act, wl.zero_frac)
    layers = []
    for spec in wl.layers:
        f = draw_weights(rng, spec)
        b = draw_bias(rng, spec)
        layers.append((f, b, spec))
    return x, layers


def next_layer_input(y_prev, spec_next):
    """Input of the next layer of a chain from the previous layer's int8
    NCHW output.  Where the next layer's image is half the size (a new
    network stage) the activations are max-pooled 2x2 with stride 2; the
    configuration names the stage sizes but not the downsampling, and
    max-pooling is exact on int8 and keeps the ReLU-like distribution."""
    n, c, h, w = y_prev.shape
    assert c == spec_next.cin, (c, spec_next.cin)
    if (h, w) == (spec_next.h, spec_next.w):
        return np.ascontiguousarray(y_prev)
    assert (h // 2, w // 2) == (spec_next.h, spec_next.w) and h % 2 == 0 and w % 2 == 0
    v = y_prev.reshape(n, c, h // 2, 2, w // 2, 2)
    return np.ascontiguousarray(v.max(axis=(3, 5)))


def random_case(seed, n, cin, cout, h, w, signed=True, zero_frac=0.0, wscale=None):
    """A generic random layer for parity sweeps: full-range int8 (or
    non-negative) activations, normal weights, bias U[-64, 64]."""
    rng = np.random.default_rng(seed)
    shape = (n, cin, h, w)
    if signed:
        x = rng.integers(-128, 128, shape).astype(np.int8)
    else:
        x = draw_activations(rng, shape, "halfnormal24", zero_frac)
    sd = np.sqrt(2.0 / (9 * cin)) if wscale is None else wscale
    f = rng.normal(0.0, sd, (cout, cin, 3, 3)).astype(np.float32)
    b = rng.integers(-64, 65, cout).astype(np.int32)
    return x, f, b
