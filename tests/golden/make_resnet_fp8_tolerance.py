"""Writes resnet_fp8_tolerance.json: the logit bound of the fp8 residual-
network parity tests, from the oracle alone.

The same model as make_fp8_tolerance.py (the fp8 matrix instruction's sums
are off by up to about 2^-16.4 of their sum of magnitudes): the oracle's fp8
residual forward with every sum moved by u EPS sum|products| (u in [-1, 1),
hashed, EPS = 2^-16) for SEEDS independent patterns, against its exact fp8
forward, on every fp8 residual parity case (tests/resnet_cases.py); the bound
is MARGIN times the largest difference.  The parity tests use it as the
logit bound and as the excuse band of the flips (sites whose oracle |logit|
is within it).

Run from the repository root:  python tests/golden/make_resnet_fp8_tolerance.py
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))                   # tests/
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))  # repository root

import oracle  # noqa: E402
from resnet_cases import RESNET_FP8_CASES, case_inputs  # noqa: E402

MARGIN = 2.0
EPS = 2.0 ** -16
SEEDS = 4


def main():
    rows = []
    for case in RESNET_FP8_CASES:
        weights, det, first, last = case_inputs(case)
        d, T, blocks, layout = case["d"], case["T"], case["blocks"], case["layout"]
        planes = oracle.unpack_paper(d, T, det, first, last) if layout == "paper" else oracle.unpack(d, T, det)
        a = oracle.forward_resnet(d, T, planes, blocks, weights, False, layout, fp8=True)
        err = np.zeros_like(a)
        for seed in range(SEEDS):
            b = oracle.forward_resnet(d, T, planes, blocks, weights, False, layout, fp8=True, fp8_sum_eps=EPS,
                                      fp8_sum_seed=seed)
            err = np.maximum(err, np.abs(a - b))
        row = dict(name=case["name"], max_abs=float(err.max()), median_abs_logit=float(np.median(np.abs(a))))
        print(row, flush=True)
        rows.append(row)
    out = dict(note="fp8 residual-network logit bound: MARGIN x the largest difference between the oracle's "
                    "exact fp8 residual forward and the same with every sum moved by up to EPS sum|products| "
                    "(SEEDS hashed patterns) over the fp8 residual parity cases",
               margin=MARGIN, eps=EPS, seeds=SEEDS,
               tol_max_abs_logit_err=MARGIN * max(r["max_abs"] for r in rows), cases=rows)
    with open(os.path.join(HERE, "resnet_fp8_tolerance.json"), "w") as f:
        json.dump(out, f, indent=1)
    print("tol", out["tol_max_abs_logit_err"])


if __name__ == "__main__":
    main()
