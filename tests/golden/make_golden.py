"""Writes tests/golden/configs.json: the oracle's results on the full-size
seeded workloads, for the GPU parity tests to compare against without
re-running the slow CPU oracle.

For C1, C2, every layer of C3 (the four-layer chain, each layer's input
being the previous layer's int8 output, max-pooled 2x2 where the next stage
halves the image), C4 and C5: the calibrated input tap exponents e_B, weight
tap exponents e_G, alignment shifts, output shift, the SHA-256 of the full
int8 output in NCHW order, and 64 sampled output values.  The same record for
F(2x2, 3x3) of each configuration's first layer goes under "f2_layers".

With ``--bits 10`` the same records for the int8/10 variant (10-bit
Winograd-domain integers, Sec. V) go to tests/golden/configs_i10.json.

Uses only the oracle and the seeded input generators.  Run from the
repository root:  python tests/golden/make_golden.py [--bits 10]
"""
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads  # noqa: E402
from oracle import quant, tapwise  # noqa: E402


def layer_record(x, f, b, spec, bits=8, m=4):
    eb = tapwise.calibrate_input_exps(x, m=m, bits=bits)
    plan0 = tapwise.make_plan(f, eb, bias=b, out_shift=0, relu=spec.relu, m=m, bits=bits)
    if spec.out_shift is None:
        z = tapwise.prequant_output(x, plan0)
        zmax = int(np.abs(z).max(initial=0))
        s = min(tapwise.OUT_SHIFT_MAX, max(0, quant.cexp(zmax)))
    else:
        s, zmax = spec.out_shift, None
    plan = tapwise.make_plan(f, eb, bias=b, out_shift=s, relu=spec.relu, m=m, bits=bits)
    y = tapwise.conv_int8(x, plan)
    rng = np.random.default_rng(1234)
    idx = [tuple(int(rng.integers(0, d)) for d in y.shape) for _ in range(64)]
    rec = {
        "shape_in": list(x.shape), "shape_out": list(y.shape), "relu": bool(spec.relu),
        "e_b": eb, "e_g": plan["e_g"], "sh": plan["sh"], "e_o": plan["e_o"], "out_shift": s,
        "zmax": zmax, "epilogue_bound": int(tapwise.epilogue_bound(plan)),
        "sha256_nchw": hashlib.sha256(np.ascontiguousarray(y).tobytes()).hexdigest(),
        "samples": [[list(i), int(y[i])] for i in idx],
        "saturated_fraction": float(np.mean(np.abs(y.astype(np.int64)) >= 127)),
    }
    return rec, y


def main():
    bits = 10 if "--bits" in sys.argv and sys.argv[sys.argv.index("--bits") + 1] == "10" else 8
    out = {}
    for name in ("C1", "C2", "C3", "C4", "C5") if bits == 8 else ("C3", "C4", "C5"):
        t0 = time.time()
        x, layers = workloads.generate(name)
        recs = []
        cur = x
        for k, (f, b, spec) in enumerate(layers):
            if k > 0:
                cur = workloads.next_layer_input(cur, spec)
            rec, y = layer_record(cur, f, b, spec, bits)
            recs.append(rec)
            cur = y
        out[name] = {"layers": recs}
        if bits == 8:
            f, b, spec = layers[0]
            out[name]["f2_layers"] = [layer_record(x, f, b, spec, bits, m=2)[0]]
        print(f"{name}: {len(recs)} layer(s) in {time.time() - t0:.1f} s", flush=True)
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)),
                        "configs.json" if bits == 8 else "configs_i10.json")
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main()
