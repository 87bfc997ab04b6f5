"""GPU parity of the input transform's two requantization forms against the
oracle, bit for bit: the one-instruction saturating form (every input
exponent e_B <= 16 - bits, the range calibration produces) at its edges
e_B = 0 and e_B = 16 - bits, and the shift-and-clamp form that serves plans
with a larger exponent, on inputs at the int8 rails (largest |V|, most
clamping) and on random ones."""
import numpy as np
import pytest

import paper_2209_12982_amd as W
import workloads
from oracle import tapwise

from gpu_util import to_device, torch_dev, workspace

pytestmark = pytest.mark.gpu

PLANS = {(4, 8): W.wino_f4_plan, (2, 8): W.wino_f2_plan, (4, 10): W.wino_f4_plan_i10, (2, 10): W.wino_f2_plan_i10}


def _exponents(kind, ntap, bits, rng):
    top = 16 - bits
    if kind == "sat_edges":
        return [0 if t % 2 == 0 else top for t in range(ntap)]
    if kind == "sat_random":
        return [int(v) for v in rng.integers(0, top + 1, ntap)]
    # one tap past the saturating form's range sends the plan to the other form
    eb = [int(v) for v in rng.integers(0, 15, ntap)]
    eb[ntap // 2] = top + 1
    return eb


@pytest.mark.parametrize("m,bits", list(PLANS))
@pytest.mark.parametrize("layout", [W.NCHW, W.NHWC])
@pytest.mark.parametrize("kind", ["sat_edges", "sat_random", "fallback"])
@pytest.mark.parametrize("rails", [True, False])
def test_input_requant_forms_bitexact(m, bits, layout, kind, rails):
    torch = torch_dev()
    n, cin, cout, h, w = 2, 70, 8, 13, 18
    rng = np.random.default_rng(600 + 10 * m + bits)
    x, f, b = workloads.random_case(601, n, cin, cout, h, w, signed=True)
    if rails:
        x = np.where(rng.random(x.shape) < 0.5, -128, 127).astype(np.int8)
    ntap = (m + 2) ** 2
    eb = _exponents(kind, ntap, bits, rng)
    gp = PLANS[(m, bits)](f, eb, bias=b)
    ws = workspace(gp, n, h, w)
    th, tw = tapwise.tile_grid(h, w, m)
    dt = torch.float16 if bits == 10 else torch.int8
    vq = torch.empty((ntap, n * th * tw, cin), dtype=dt, device="cuda")
    W.wino_f4_debug_input_transform(gp, to_device(x, layout), n, h, w, layout, vq, ws)
    torch.cuda.synchronize()
    got = vq.cpu().numpy().astype(np.int64)
    ref = tapwise.input_taps_quantized(x, eb, m=m, bits=bits)
    assert (got == ref).all(), f"{(got != ref).sum()} mismatches"
    if rails and kind == "sat_edges" and (m == 4 or bits == 8):       # F2's |V| <= 510 stays inside 10 bits
        lim = 2 ** (bits - 1)
        assert (ref == lim - 1).any() and (ref == -lim).any()      # both rails reached
