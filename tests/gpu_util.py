"""Helpers for GPU parity tests: device placement and layout conversion only
(no method arithmetic)."""
import numpy as np

import paper_2209_12982_amd as W


def torch_dev():
    import torch
    if not torch.cuda.is_available():
        import pytest
        pytest.skip("no GPU")
    return torch


def to_device(x_nchw, layout):
    torch = torch_dev()
    a = np.asarray(x_nchw, dtype=np.int8)
    if layout == W.NHWC:
        a = np.ascontiguousarray(a.transpose(0, 2, 3, 1))
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def from_device_nchw(t, layout):
    a = t.cpu().numpy()
    if layout == W.NHWC:
        a = a.transpose(0, 3, 1, 2)
    return np.ascontiguousarray(a)


def empty_out(n, c, h, w, layout):
    torch = torch_dev()
    shape = (n, c, h, w) if layout == W.NCHW else (n, h, w, c)
    return torch.full(shape, 77, dtype=torch.int8, device="cuda")   # poison value


def workspace(plan, n, h, w, variant=W.SPLIT):
    torch = torch_dev()
    nb = W.wino_f4_workspace_bytes(plan, n, h, w, variant)
    return torch.empty(max(nb, 1), dtype=torch.int8, device="cuda")


def run_conv(plan, x_nchw, layout, variant=W.SPLIT):
    torch = torch_dev()
    n, cin, h, w = x_nchw.shape
    x = to_device(x_nchw, layout)
    y = empty_out(n, plan.cout, h, w, layout)
    ws = workspace(plan, n, h, w, variant) if variant == W.SPLIT else None
    W.wino_f4_conv_int8(plan, x, y, n, h, w, layout, variant, ws)
    torch.cuda.synchronize()
    return from_device_nchw(y, layout)
