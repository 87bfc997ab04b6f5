"""Prints the weight-quantization study table of oracle/quant_study.py: mean
log2 relative error of the spatial weights, all 3x3 layers of C1-C5 pooled,
for the paper's procedure (per-group mean, standard deviation and searched
scale; Winograd-domain weights back-projected) and the library's scheme
(power-of-two max-abs scales), on the synthetic weights as drawn and with
per-channel log-normal scales.  Run from the repository root:
    python tests/quant_study_report.py        (a few minutes)"""
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import workloads  # noqa: E402
from oracle import quant_study as qs  # noqa: E402


def layers(scaled):
    out = []
    for name in ("C1", "C2", "C3", "C4", "C5"):
        _, ls = workloads.generate(name)
        out += [f for f, _, _ in ls]
    if scaled:
        out = [workloads.channel_scaled(f, 100 + i) for i, f in enumerate(out)]
    return out


res = {}
for scaled in (False, True):
    for m in (4, 2):
        res[(scaled, m)] = qs.study(layers(scaled), m=m)
        print(f"# done: scaled={scaled} F{m}", file=sys.stderr, flush=True)

rows = [("spatial", "layer"), ("spatial", "channel")] + [("winograd", st) for st in qs.STRATEGIES]
print("| domain | grouping | paper, i.i.d. | paper, channel-scaled | pow2, i.i.d. | pow2, channel-scaled |")
print("|---|---|---|---|---|---|")
for m in (4, 2):
    for dom, st in rows:
        if dom == "spatial" and m == 2:
            continue
        cells = [f"2^{qs.mean_log2(res[(sc, m)], dom, st, sch):.2f}"
                 for sch in ("paper", "pow2") for sc in (False, True)]
        name = "spatial" if dom == "spatial" else f"F{m} Winograd"
        print(f"| {name} | {st.replace('_', ' & ')} | " + " | ".join(cells) + " |")
n = int(np.sum([np.asarray(f).size for f in layers(False)]))
print(f"\n{n} weights in {len(layers(False))} layers")
