"""Writes resnet_tolerance.json: the logit bound of the bf16 residual-network
parity tests, from the oracle alone.

In a residual network the shortcuts carry each block's output forward
without the squashing of a plain chain, so an activation that two valid fp32
summations round to neighbouring bf16 values moves the logits further than
in the plain networks (whose bound is 2e-2).  On every residual parity case
(tests/resnet_cases.py) this records the largest logit difference between
the oracle's bf16 forward with fp64 and with fp32 sums; the bound is MARGIN
times the largest, and never below the plain bound.

Run from the repository root:  python tests/golden/make_resnet_tolerance.py
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))                   # tests/
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))  # repository root

import oracle  # noqa: E402
from resnet_cases import RESNET_CASES, case_inputs  # noqa: E402

MARGIN = 2.0
PLAIN = 2e-2


def main():
    rows = []
    for case in RESNET_CASES:
        weights, det, first, last = case_inputs(case)
        d, T, blocks, layout = case["d"], case["T"], case["blocks"], case["layout"]
        planes = oracle.unpack_paper(d, T, det, first, last) if layout == "paper" else oracle.unpack(d, T, det)
        a = oracle.forward_resnet(d, T, planes, blocks, weights, True, layout)
        b = oracle.forward_resnet(d, T, planes, blocks, weights, True, layout, acc32=True)
        row = dict(name=case["name"], max_abs=float(np.abs(a - b).max()),
                   median_abs_logit=float(np.median(np.abs(a))))
        print(row, flush=True)
        rows.append(row)
    out = dict(note="bf16 residual-network logit bound: max(2e-2, MARGIN x the largest difference between the "
                    "oracle's bf16 forward with fp64 and with fp32 sums over the residual parity cases)",
               margin=MARGIN, tol_max_abs_logit_err=max(PLAIN, MARGIN * max(r["max_abs"] for r in rows)),
               cases=rows)
    with open(os.path.join(HERE, "resnet_tolerance.json"), "w") as f:
        json.dump(out, f, indent=1)
    print("tol", out["tol_max_abs_logit_err"])


if __name__ == "__main__":
    main()
