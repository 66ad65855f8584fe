"""GPU tests of the temporal window driver (Sec. VI, parallel windows in
time) through the C ABI: stitched flips and residual of a long stream against
the oracle's single run over the whole stream (parity rule; the windows'
cores are exact because the buffer covers the receptive field), against the
GPU's own single run over the whole stream, in both layouts (with the
preparation and measurement bases at the stream's ends), several streams at
once, a length that is not a multiple of the core, and the fp8 path."""
import numpy as np
import pytest

import oracle
import paper_2604_12841_amd as pdx
from paper_2604_12841_amd import workload
from parity import TOL, _padding_zero, assert_parity, compare, dev_u64, host_u64, run_gpu, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda")


def _stream_gpu(weights, d, n, layers, core, buffer, det, dtype="bf16", layout="plaquette", first=None, last=None):
    s = pdx.Stream(weights, d, n, layers, core, buffer, dtype, n_streams=det.shape[0], layout=layout, first=first,
                   last=last)
    ddet = dev_u64(det)
    flips = torch.full((det.shape[0], s.flip_words), -1, dtype=torch.int64, device="cuda")
    res = torch.full((det.shape[0], s.det_words), -1, dtype=torch.int64, device="cuda")
    s.run(ddet, flips, res)
    torch.cuda.synchronize()
    s.close()
    return host_u64(flips), host_u64(res)


CASES = [
    dict(name="plaq_d5_n40", d=5, n=40, core=5, buffer=5, layout="plaquette", layers=workload.layer_spec(4, 64), B=2),
    dict(name="plaq_d5_n37_ragged", d=5, n=37, core=5, buffer=5, layout="plaquette",
         layers=workload.layer_spec(3, 64), B=1),
    dict(name="paper_d5_n31", d=5, n=31, core=5, buffer=5, layout="paper",
         layers=workload.paper_layer_spec([64, 64, 4], [3, 3, 3]), B=2, first="Z", last="Z"),
    dict(name="paper_d7_n28_xbasis", d=7, n=28, core=7, buffer=7, layout="paper",
         layers=workload.paper_model_layers(1), B=1, first="X", last="X"),
]


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_stream_against_oracle_whole_stream(cuda, case):
    d, n, layers, layout = case["d"], case["n"], case["layers"], case["layout"]
    weights = workload.he_normal_weights(layers, 71)
    det, _ = workload.make_inputs(d, n, case["B"], 0.01, 0.01, 72)
    first, last = case.get("first"), case.get("last")
    say("stream", case["name"], "windows", len(pdx.stream_windows(n, case["core"], case["buffer"])))
    flips, res = _stream_gpu(weights, d, n, layers, case["core"], case["buffer"], det, layout=layout, first=first,
                             last=last)
    ref = oracle.run(d, n, det, layers, weights, bf16=True, layout=layout, first=first, last=last)
    st = compare(d, n, "bf16", *ref, flips, res, layout=layout)
    say("  stats", st)
    assert_parity(st, "bf16")
    np.testing.assert_array_equal(res, oracle.residual_from_flips(d, n, det, flips))


def test_stream_against_gpu_whole_stream_d13_1000_rounds(cuda):
    """Model 1 of Table models, d = 13, 1000 rounds, core = buffer = d (the
    paper's d x d x 3d blocks), two streams: the stitched flips equal the
    GPU's single run over all 1000 rounds up to its excused sites."""
    d, n = 13, 1000
    layers = workload.paper_model_layers(1)
    weights = workload.he_normal_weights(layers, 4001)
    det, _ = workload.make_inputs(d, n, 2, 0.003, 0.003, 73)
    flips, res = _stream_gpu(weights, d, n, layers, d, d, det, layout="paper", first="Z", last="Z")
    pre = pdx.Predecoder(weights, d, n, layers, "bf16", max_batch=2, layout="paper", first="Z", last="Z")
    f1, r1, l1 = run_gpu(pre, det)
    pre.close()
    st = compare(d, n, "bf16", l1.astype(np.float64), f1, r1, flips, res, layout="paper")
    say("  against the whole-stream run", st)
    assert_parity(st, "bf16")
    assert _padding_zero(flips, n * (3 * d * d - 1)) and _padding_zero(res, n * (d * d - 1))


def test_stream_fp8(cuda):
    d, n = 5, 30
    layers = workload.paper_layer_spec([64, 64, 4], [3, 3, 3])
    weights = workload.he_normal_weights(layers, 74)
    det, _ = workload.make_inputs(d, n, 2, 0.01, 0.01, 75)
    flips, res = _stream_gpu(weights, d, n, layers, 5, 5, det, dtype="fp8", layout="paper", first="Z", last="Z")
    pre = pdx.Predecoder(weights, d, n, layers, "fp8", max_batch=2, layout="paper", first="Z", last="Z")
    f1, r1, l1 = run_gpu(pre, det)
    pre.close()
    # the whole-stream run's logits decide which sites may differ
    st = compare(d, n, "bf16", l1.astype(np.float64), f1, r1, flips, res, layout="paper", tol=TOL["fp8"])
    say("  fp8 against the whole-stream run", st)
    assert st["flip_mismatch"] == 0 and st["res_mismatch"] == 0
    np.testing.assert_array_equal(res, oracle.residual_from_flips(d, n, det, flips))
