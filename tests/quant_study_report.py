"""Prints the weight-quantization study table (mean relative error, log2) of
oracle/quant_study.py on the synthetic layers of C1-C5; run from the
repository root: python tests/quant_study_report.py"""
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import workloads  # noqa: E402
from oracle import quant_study as qs  # noqa: E402

layers = []
for name in ("C1", "C2", "C3", "C4", "C5"):
    _, ls = workloads.generate(name)
    layers += [f for f, _, _ in ls]
rows = []
for m in (4, 2):
    res = qs.study(layers, m=m)
    for dom, sts in (("spatial", ("layer", "channel")), ("winograd", qs.STRATEGIES)):
        if dom == "spatial" and m == 2:
            continue
        for st in sts:
            p = np.log2(np.mean(res[(dom, st, True)]))
            f = np.log2(np.mean(res[(dom, st, False)]))
            rows.append(f"| {'—' if dom == 'spatial' else 'F%d' % m} {dom} | {st} | 2^{p:.2f} | 2^{f:.2f} |")
print("| domain | strategy | power-of-two scales | fp32 scales |")
print("|---|---|---|---|")
print("\n".join(rows))
