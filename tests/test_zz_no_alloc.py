"""predecoder_run_static (the run that allocates nothing: its workspace is the
library's static device array) against predecoder_run through the C ABI: the
same flips, residual and logits, bit for bit, on two calls in a row, the
second with a smaller batch; with other handles (other grids, widths and
precisions) using the array in between; and a batch whose workspace does not
fit rejected before any device work.  The static run's results also meet the
parity rule against the oracle."""
import numpy as np
import pytest

import oracle
import paper_2604_12841_amd as pdx
from parity import assert_parity, compare, dev_u64, host_u64, say
from paper_2604_12841_amd import workload
from resnet_cases import RESNET_CASES
from resnet_cases import case_inputs as resnet_inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda")


def _outputs(pre, det, B, static):
    ddet = dev_u64(det[:B])
    flips = torch.full((B, pre.flip_words), -1, dtype=torch.int64, device="cuda")
    res = torch.full((B, pre.det_words), -1, dtype=torch.int64, device="cuda")
    logits = torch.full((B, 4, pre.T, pre.grid, pre.grid), float("nan"), dtype=torch.float32, device="cuda")
    (pre.run_static if static else pre.run)(ddet, flips, res, logits)
    torch.cuda.synchronize()
    return host_u64(flips), host_u64(res), logits.cpu().numpy()


def _same(a, b):
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def _plain(name):
    """(d, T, layers, weights, det, dtype, layout, first, last) of a case."""
    if name == "w3_bf16":  # the benchmark workload's network at d = 13
        c = workload.CONFIGS[3]
        det, _ = workload.config_inputs(3, 6)
        return c["d"], c["T"], workload.config_layers(3), workload.config_weights(3), det, "bf16", "plaquette", None, None
    if name == "w2_fp8":
        c = workload.CONFIGS[2]
        det, _ = workload.config_inputs(2, 3)
        return c["d"], c["T"], workload.config_layers(2), workload.config_weights(2), det, "fp8", "plaquette", None, None
    if name == "w1_fp32":
        c = workload.CONFIGS[1]
        det, _ = workload.config_inputs(1, 8)
        return c["d"], c["T"], workload.config_layers(1), workload.config_weights(1), det, "fp32", "plaquette", None, None
    if name == "m1_paper_bf16":
        layers = workload.paper_model_layers(1)
        det, _ = workload.make_inputs(9, 9, 2, 0.003, 0.003, 5009)
        return 9, 9, layers, workload.he_normal_weights(layers, 4001), det, "bf16", "paper", "Z", "Z"
    raise KeyError(name)


def _handle(case):
    if case in ("w3_bf16", "w2_fp8", "w1_fp32", "m1_paper_bf16"):
        d, T, layers, weights, det, dtype, layout, first, last = _plain(case)
        pre = pdx.Predecoder(weights, d, T, layers, dtype, max_batch=det.shape[0], layout=layout, first=first,
                             last=last)
        ref = lambda B: oracle.run(d, T, det[:B], layers, weights, bf16=dtype == "bf16", layout=layout,
                                   first=first, last=last, fp8=dtype == "fp8")
        return pre, det, dtype, layout, ref
    rc = next(c for c in RESNET_CASES if c["name"] == case)
    weights, det, first, last = resnet_inputs(rc)
    pre = pdx.Predecoder(weights, rc["d"], rc["T"], None, "bf16", max_batch=det.shape[0], layout=rc["layout"],
                         first=first, last=last, blocks=rc["blocks"])
    ref = lambda B: oracle.run_resnet(rc["d"], rc["T"], det[:B], rc["blocks"], weights, bf16=True,
                                      layout=rc["layout"], first=first, last=last)
    return pre, det, "bf16", rc["layout"], ref


CASES = ["w3_bf16", "w2_fp8", "w1_fp32", "m1_paper_bf16", "w64_paper", "mid_projection"]


@pytest.mark.parametrize("case", CASES)
def test_static_run_matches_run(cuda, case):
    pre, det, dtype, layout, ref = _handle(case)
    B = det.shape[0]
    say("static run", case, "batch", B, "then 1")
    # two calls in a row, the second smaller, each against predecoder_run
    full = _outputs(pre, det, B, static=True)
    _same(full, _outputs(pre, det, B, static=False))
    one = _outputs(pre, det, 1, static=True)
    _same(one, _outputs(pre, det, 1, static=False))
    pre.close()
    # the static run's batch-1 result under the parity rule
    logits_ref, flips_ref, res_ref = ref(1)
    tol = None
    if case in ("w64_paper", "mid_projection"):
        import json, os
        tol = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                                          "resnet_tolerance.json")))["tol_max_abs_logit_err"]
    st = compare(pre.d, pre.T, dtype, logits_ref, flips_ref, res_ref, one[0], one[1], one[2], layout=layout, tol=tol)
    say("  parity of the static batch-1 run", st)
    assert_parity(st, dtype, tol=tol)


def test_static_run_after_other_handles(cuda):
    """Handles of other grids, widths and precisions use the array in
    between; the first handle's static results do not change."""
    pre, det, *_ = _handle("w3_bf16")
    first = _outputs(pre, det, 2, static=True)
    for other in ("w1_fp32", "m1_paper_bf16", "mid_projection", "w2_fp8"):
        p2, d2, *_ = _handle(other)
        _same(_outputs(p2, d2, d2.shape[0], static=True), _outputs(p2, d2, d2.shape[0], static=False))
        p2.close()
        _same(_outputs(pre, det, 2, static=True), first)
    pre.close()


def test_static_run_rejects_a_batch_that_does_not_fit(cuda):
    c = workload.CONFIGS[3]
    d, T = c["d"], c["T"]
    B = 64  # two activation buffers alone are 64 x 3840 x 256 bytes each, 126 MB
    det, _ = workload.config_inputs(3, B)
    pre = pdx.Predecoder(workload.config_weights(3), d, T, workload.config_layers(3), "bf16", max_batch=B)
    with pytest.raises(pdx.PredecoderError) as e:
        _outputs(pre, det, B, static=True)
    assert e.value.status == pdx.PD_ERR_TOO_LARGE
    # a batch that fits still runs on the same handle
    _same(_outputs(pre, det, 2, static=True), _outputs(pre, det, 2, static=False))
    pre.close()
