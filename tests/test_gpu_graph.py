"""Recorded runs (HIP graphs) through the C ABI: every replay equals an eager
predecoder_run on the same input bit for bit, over several replays with
eager work, synchronisation and new input data in between; bf16 (batch 1
with split K loops, and a larger batch), fp8, a residual network, and a
network that reuses activation buffers at other row widths (the clearing
kernel inside the graph)."""
import numpy as np
import pytest

import paper_2604_12841_amd as pdx
from paper_2604_12841_amd import workload
from parity import dev_u64, host_u64, run_gpu, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

G = workload.GELU_TANH
CASES = [
    dict(name="m1_paper_b1", layers=workload.paper_model_layers(1), d=7, B=1, dtype="bf16", layout="paper"),
    dict(name="plaq_b16", layers=workload.layer_spec(3, 128), d=9, B=16, dtype="bf16", layout="plaquette"),
    dict(name="fp8_b2", layers=workload.paper_model_layers(4), d=5, B=2, dtype="fp8", layout="paper"),
    dict(name="widths_b3", layers=[(2, 64, 3, G), (64, 128, 3, G), (128, 128, 3, G), (128, 64, 3, G),
                                   (64, 4, 1, workload.NONE)], d=5, B=3, dtype="bf16", layout="plaquette"),
    dict(name="resnet_b1", blocks=workload.resnet_blocks([64, 128, 128]), d=5, B=1, dtype="bf16", layout="paper"),
]


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda")


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_graph_replays_equal_eager_runs(cuda, case):
    d = T = case["d"]
    B, layout = case["B"], case["layout"]
    first = last = "Z" if layout == "paper" else None
    if "blocks" in case:
        weights = workload.resnet_weights(case["blocks"], 95)
        pre = pdx.Predecoder(weights, d, T, None, case["dtype"], max_batch=B, layout=layout, first=first,
                             last=last, blocks=case["blocks"])
    else:
        weights = workload.he_normal_weights(case["layers"], 95)
        pre = pdx.Predecoder(weights, d, T, case["layers"], case["dtype"], max_batch=B, layout=layout,
                             first=first, last=last)
    say("graph", case["name"])
    ddet = dev_u64(workload.make_inputs(d, T, B, 0.01, 0.01, 96)[0])
    flips = torch.zeros((B, pre.flip_words), dtype=torch.int64, device="cuda")
    res = torch.zeros((B, pre.det_words), dtype=torch.int64, device="cuda")
    logits = torch.zeros((B, 4, T, pre.grid, pre.grid), dtype=torch.float32, device="cuda")
    g = pre.graph(ddet, flips, res, logits)
    other = pdx.Predecoder(workload.he_normal_weights(workload.layer_spec(2, 64), 97), 5, 3,
                           workload.layer_spec(2, 64), "bf16", max_batch=2)
    odet = workload.make_inputs(5, 3, 2, 0.02, 0.02, 98)[0]
    for rep in range(4):
        det = workload.make_inputs(d, T, B, 0.01, 0.01, 100 + rep)[0]
        ddet.copy_(dev_u64(det))  # new input in the recorded buffer
        for t in (flips, res):
            t.fill_(-1)
        logits.fill_(float("nan"))
        g.launch()
        torch.cuda.synchronize()
        gf, gr, gl = host_u64(flips), host_u64(res), logits.cpu().numpy()
        run_gpu(other, odet)  # eager work of another handle in between
        ef, er, el = run_gpu(pre, det)  # eager run of the same handle on the same input
        assert (gf == ef).all() and (gr == er).all() and np.array_equal(gl, el), (case["name"], rep)
    g.close()
    pre.close()
    other.close()

