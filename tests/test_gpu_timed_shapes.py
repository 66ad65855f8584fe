"""GPU parity at the shapes the committed timing profiles measure: Models 1
to 5 of Table models in the paper's layout at 13^3, 21^3 and 31^3
(batch 1, where the K loops are split, and batch 64), in bf16 and, for
Models 1, 2, 4 and 5, in fp8; Model 6 at 13^3, 21^3 and 31^3 (batch 1 and
16) in bf16 and fp8.  Each
run is the launch configuration the benchmark times (one handle, the whole
batch); sampled samples (first and last) are compared with the oracle under
the parity rule of parity.py, every sample's residual with the oracle's
residual of the GPU's flips, and every sample's flips and residual with the
threshold of the GPU's own logits.  Also the two plaquette-grid networks of
the d = 5 ... 31 sweep: at batch 1 (the latency rows, where layers run as
output slices or split K loops, the head layer included), and batched at the
d that the benchmark workloads do not cover."""
import json
import os

import numpy as np
import pytest

import oracle
import paper_2604_12841_amd as pdx
from parity import TOL, assert_flips_follow_logits, assert_parity, compare, run_gpu, say
from paper_2604_12841_amd import workload

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

RESNET_TOL = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                                         "resnet_tolerance.json")))["tol_max_abs_logit_err"]


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda")


def _inputs(d, B):
    # the benchmark's paper-model inputs: p = q = 0.003, noise seed 5000 + d
    det, _ = workload.make_inputs(d, d, B, 0.003, 0.003, 5000 + d)
    return det


def _check(d, T, dtype, det, rows, flips, res, logits, ref, tol):
    B = det.shape[0]
    st = compare(d, T, dtype, *ref, flips[rows], res[rows], logits[rows], layout="paper", tol=tol)
    say("  samples", rows, "of", B, st)
    assert_parity(st, dtype, tol=tol)
    np.testing.assert_array_equal(res, oracle.residual_from_flips(d, T, det, flips))
    assert_flips_follow_logits(d, T, det, logits, flips, res, layout="paper")


CASES = [(m, d, b, dt) for dt in ("bf16", "fp8") for m in (1, 2, 3, 4, 5) for d in (13, 21, 31) for b in (1, 64)
         if dt == "bf16" or m != 3]


@pytest.mark.parametrize("model,d,batch,dtype", CASES, ids=["m%d_d%d_b%d_%s" % c for c in CASES])
def test_paper_model_at_timed_shape(cuda, model, d, batch, dtype):
    T = d
    layers = workload.paper_model_layers(model)
    weights = workload.he_normal_weights(layers, 4000 + model)  # the benchmark's weights
    det = _inputs(d, batch)
    rows = [0] if batch == 1 else [0, batch - 1]
    say("Model", model, "d = T =", d, "batch", batch, dtype)
    pre = pdx.Predecoder(weights, d, T, layers, dtype, max_batch=batch, layout="paper", first="Z", last="Z")
    flips, res, logits = run_gpu(pre, det)
    pre.close()
    ref = oracle.run(d, T, det[rows], layers, weights, bf16=dtype == "bf16", layout="paper", first="Z", last="Z",
                     fp8=dtype == "fp8")
    _check(d, T, dtype, det, rows, flips, res, logits, ref, TOL[dtype])


RESNET_FP8_TOL = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                                             "resnet_fp8_tolerance.json")))["tol_max_abs_logit_err"]
M6_CASES = [(d, b, dt) for dt in ("bf16", "fp8") for d in (13, 21, 31) for b in (1, 16)]


@pytest.mark.parametrize("d,batch,dtype", M6_CASES, ids=["d%d_b%d_%s" % c for c in M6_CASES])
def test_model6_at_timed_shape(cuda, d, batch, dtype):
    T = d
    blocks = workload.MODEL6_BLOCKS
    weights = workload.resnet_weights(blocks, 4006)  # the benchmark's weights
    det = _inputs(d, batch)
    rows = [0] if batch == 1 else [0, batch - 1]
    say("Model 6 d = T =", d, "batch", batch, dtype)
    pre = pdx.Predecoder(weights, d, T, None, dtype, max_batch=batch, layout="paper", first="Z", last="Z",
                         blocks=blocks)
    flips, res, logits = run_gpu(pre, det)
    pre.close()
    ref = oracle.run_resnet(d, T, det[rows], blocks, weights, bf16=dtype == "bf16", layout="paper", first="Z",
                            last="Z", fp8=dtype == "fp8")
    _check(d, T, dtype, det, rows, flips, res, logits, ref, RESNET_TOL if dtype == "bf16" else RESNET_FP8_TOL)



@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_model6_batch_and_its_sub_batches(cuda, dtype):
    """Model 6 at 13^3, batch 16, whose units overfill the chip's workgroup
    slots by a short remainder: the last samples then run as a sub-batch of
    their own with split K loops.  Some split point b must exist such that
    samples [0, b) run alone give exactly the batch's flips, residual and
    logits (the same unsplit launches), and samples [b, 16) run alone agree
    with the batch's within the logit tolerance, flips and residual exact
    outside its band (alone, they may split their K loops differently)."""
    d = T = 13
    batch = 16
    blocks = workload.MODEL6_BLOCKS
    weights = workload.resnet_weights(blocks, 4006)
    det = _inputs(d, batch)
    tol = RESNET_TOL if dtype == "bf16" else RESNET_FP8_TOL
    say("Model 6 sub-batches, d = T =", d, "batch", batch, dtype)
    pre = pdx.Predecoder(weights, d, T, None, dtype, max_batch=batch, layout="paper", first="Z", last="Z",
                         blocks=blocks)
    flips, res, logits = run_gpu(pre, det)
    found = None
    for b in range(batch - 1, 0, -1):
        if all(np.array_equal(x, z[:b]) for x, z in zip(run_gpu(pre, det[:b]), (flips, res, logits))):
            found = b
            break
    assert found is not None
    f2, r2, l2 = run_gpu(pre, det[found:])
    pre.close()
    st = compare(d, T, dtype, logits[found:].astype(np.float64), flips[found:], res[found:], f2, r2, l2,
                 layout="paper", tol=tol)
    say("  first", found, "samples exact; the rest alone against the batch:", st)
    assert_parity(st, dtype, tol=tol)


SWEEP_B1 = [(w, d, dt) for dt in ("bf16", "fp8") for w in (3, 4) for d in (5, 7, 9, 13, 17, 21, 25, 31)]


@pytest.mark.parametrize("wl,d,dtype", SWEEP_B1, ids=["w%d_d%d_b1_%s" % c for c in SWEEP_B1])
def test_plaquette_network_at_batch_one(cuda, wl, d, dtype):
    """The sweep's batch-1 runs (`bench.py --workload W --d D --batch 1`):
    the workload's network and weights, its noise, d = T."""
    c = workload.CONFIGS[wl]
    layers = workload.config_layers(wl)
    weights = workload.config_weights(wl)
    det, _ = workload.make_inputs(d, d, 1, c["p"], c["q"], 2000 + wl)
    say("workload", wl, "network at d = T =", d, "batch 1", dtype)
    pre = pdx.Predecoder(weights, d, d, layers, dtype, max_batch=1)
    flips, res, logits = run_gpu(pre, det)
    pre.close()
    ref = oracle.run(d, d, det, layers, weights, bf16=dtype == "bf16", fp8=dtype == "fp8")
    st = compare(d, d, dtype, *ref, flips, res, logits, tol=TOL[dtype])
    say("  stats", st)
    assert_parity(st, dtype, tol=TOL[dtype])
    np.testing.assert_array_equal(res, oracle.residual_from_flips(d, d, det, flips))
    assert_flips_follow_logits(d, d, det, logits, flips, res)


SWEEP_BATCHED = [(w, d, dt) for dt in ("bf16", "fp8") for w in (3, 4) for d in (5, 7, 9, 17, 21, 25)]


def sweep_batch(d):
    # the sweep's batch: about the d = 13, batch 4096 voxel count per step
    return max(16, round(4096 * 13 * 14 * 14 / (d * (d + 1) ** 2)))


@pytest.mark.parametrize("wl,d,dtype", SWEEP_BATCHED, ids=["w%d_d%d_%s" % c for c in SWEEP_BATCHED])
def test_plaquette_network_batched_at_sweep_shape(cuda, wl, d, dtype):
    """The sweep's batched runs (`bench.py --workload W --d D --batch B`, B
    from sweep_batch): the first and the last sample against the oracle."""
    c = workload.CONFIGS[wl]
    layers = workload.config_layers(wl)
    weights = workload.config_weights(wl)
    B = sweep_batch(d)
    det, _ = workload.make_inputs(d, d, B, c["p"], c["q"], 2000 + wl)
    rows = [0, B - 1]
    say("workload", wl, "network at d = T =", d, "batch", B, dtype)
    pre = pdx.Predecoder(weights, d, d, layers, dtype, max_batch=B)
    flips, res, logits = run_gpu(pre, det)
    pre.close()
    ref = oracle.run(d, d, det[rows], layers, weights, bf16=dtype == "bf16", fp8=dtype == "fp8")
    st = compare(d, d, dtype, *ref, flips[rows], res[rows], logits[rows], tol=TOL[dtype])
    say("  samples", rows, "stats", st)
    assert_parity(st, dtype, tol=TOL[dtype])
    np.testing.assert_array_equal(res, oracle.residual_from_flips(d, d, det, flips))
    assert_flips_follow_logits(d, d, det, logits, flips, res)
