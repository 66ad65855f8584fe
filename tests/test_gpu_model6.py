"""GPU parity of residual networks (Model 6, Sec. VI, Fig.
Model8Representation) against the oracle's residual forward in bf16 mode,
through the C ABI: Model 6 itself on small volumes, projections in a middle
block (widening and narrowing, which also reuse activation buffers at other
row widths), 256-wide slices, ReLU and linear blocks, both layouts, batch 1
(split K loops) and larger batches.  Logits within the bound that
tests/golden/make_resnet_tolerance.py derives from the oracle alone; flips
and residual bits exact outside the sites that bound excuses."""
import json
import os

import pytest

import oracle
import paper_2604_12841_amd as pdx
from parity import assert_parity, compare, run_gpu, say
from resnet_cases import RESNET_CASES, case_inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                                  "resnet_tolerance.json")))["tol_max_abs_logit_err"]


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda")


@pytest.mark.parametrize("case", RESNET_CASES, ids=[c["name"] for c in RESNET_CASES])
def test_resnet_parity(cuda, case):
    blocks, d, T, B, layout = case["blocks"], case["d"], case["T"], case["B"], case["layout"]
    weights, det, first, last = case_inputs(case)
    say("resnet", case["name"], "blocks", blocks, "d", d, "T", T, "B", B)
    pre = pdx.Predecoder(weights, d, T, None, "bf16", max_batch=B, layout=layout, first=first, last=last,
                         blocks=blocks)
    flips, res, logits = run_gpu(pre, det)
    assert pre.num_stages == len(blocks) + 2
    # a second run on the same handle (buffers now hold the first run's rows)
    f2, r2, l2 = run_gpu(pre, det)
    pre.close()
    ref = oracle.run_resnet(d, T, det, blocks, weights, bf16=True, layout=layout, first=first, last=last)
    st = compare(d, T, "bf16", *ref, flips, res, logits, layout=layout, tol=TOL)
    say("  stats", st)
    assert_parity(st, "bf16", tol=TOL)
    assert (flips == f2).all() and (res == r2).all() and (logits == l2).all()
