"""GPU parity of the fp8 path (E4M3 weights and activations with fp32
accumulation, the precision the paper deploys in, Sec. VI) against the
oracle's fp8 mode, through the C ABI, under the fp8 parity rule of
parity.py: the fp8 parity cases (benchmark workloads 2 and 3, ReLU, and
Models 1, 2, 4 and 5 of Table models in the paper's layout), the benchmark's
full d = 13 batch in its launch configuration (sampled samples), the same
samples in a small batch (split K loops), run-to-run determinism, and tight
per-site checks of the fp8 output layer and of an fp8 hidden layer with the
fused head."""
import numpy as np
import pytest

import oracle
import paper_2604_12841_amd as pdx
from fp8_cases import FP8_CASES, case_inputs
from paper_2604_12841_amd import workload
import tight
from parity import _padding_zero, assert_parity, compare, config_case, run_gpu, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda")


def _gpu(d, T, layers, weights, det, layout, first, last, max_batch=None):
    pre = pdx.Predecoder(weights, d, T, layers, "fp8", max_batch=max_batch or det.shape[0], layout=layout,
                         first=first, last=last)
    out = run_gpu(pre, det)
    pre.close()
    return out


@pytest.mark.parametrize("case", FP8_CASES, ids=[c["name"] for c in FP8_CASES])
def test_fp8_parity(cuda, case):
    d, T, layers, weights, det, layout, first, last = case_inputs(case)
    say("fp8 case", case["name"], "d", d, "T", T, "B", det.shape[0], "layers", layers)
    flips, res, logits = _gpu(d, T, layers, weights, det, layout, first, last)
    ref = oracle.run(d, T, det, layers, weights, bf16=False, layout=layout, first=first, last=last, fp8=True)
    st = compare(d, T, "fp8", *ref, flips, res, logits, layout=layout)
    say("  stats", st)
    assert_parity(st, "fp8")


@pytest.mark.parametrize("cfg", [3, 5])
def test_fp8_full_size_sampled(cuda, cfg):
    """Workloads 3 (d = T = 13, batch 4096, flat tiles) and 5 (d = T = 31,
    batch 256, box tiles), 8 x 128, at their full batch in fp8: three samples
    against the oracle, every sample's residual against the oracle's residual
    of the GPU flips; then the same samples alone (a small batch, whose K
    loops are split) against the full batch."""
    d, T, _, layers, weights, det, _ = config_case(cfg)
    B = det.shape[0]
    idx = [0, B // 2, B - 1]
    say("fp8 full size d", d, "T", T, "B", B)
    flips, res, logits = _gpu(d, T, layers, weights, det, "plaquette", None, None)
    np.testing.assert_array_equal(res, oracle.residual_from_flips(d, T, det, flips))
    assert _padding_zero(flips, T * (3 * d * d - 1)) and _padding_zero(res, T * (d * d - 1))
    assert np.isfinite(logits).all()
    ref = oracle.run(d, T, det[idx], layers, weights, bf16=False, fp8=True)
    st = compare(d, T, "fp8", *ref, flips[idx], res[idx], logits[idx])
    say("  stats", st)
    assert_parity(st, "fp8")
    f2, r2, l2 = _gpu(d, T, layers, weights, det[idx], "plaquette", None, None)
    st2 = compare(d, T, "fp8", logits[idx].astype(np.float64), flips[idx], res[idx], f2, r2, l2)
    say("  small batch against the full batch", st2)
    assert_parity(st2, "fp8")


def test_fp8_deterministic(cuda):
    d, T, layers, weights, det, layout, first, last = case_inputs(FP8_CASES[3])
    a = _gpu(d, T, layers, weights, det, layout, first, last)
    b = _gpu(d, T, layers, weights, det, layout, first, last)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


# ---- tight checks of every fp8 layer -------------------------------------
#
# predecoder_activations gives each hidden layer's E4M3 output.  Layer by
# layer, the test recomputes the layer in fp64 from the GPU's own input (the
# planes for layer 1, else the previous layer's GPU codes) with the oracle's
# quantisation points, under the rule of tight.py: every output code must
# equal the expected one, except where the GPU's summation error (EPS_MM x
# sum|products| for the fp8 instruction, EPS_32 for layer 1's bf16 one) or
# its activation arithmetic can move the value across an E4M3 rounding
# boundary; there the code must be one of the codes reachable within those
# bounds.  The logits are then checked from the GPU's last hidden codes to
# the bound of their own sums, with nothing excused.
EPS_MM = 2.0 ** -16 + 2.0 ** -18
EPS_32 = 2.0 ** -17


def _q8(t):
    return tight.q_e4m3(t)


def _layer_weights(weights, layers):
    """Per layer: (E4M3-valued weights x scales, bias) as fp64 tensors."""
    out, off = [], 0
    for ci, co, k, act in layers:
        nw = co * ci * k ** 3
        w = torch.from_numpy(weights[off:off + nw].reshape(co, ci, k, k, k).astype(np.float64))
        b = torch.from_numpy(weights[off + nw:off + nw + co].astype(np.float64))
        off += nw + co
        e = torch.tensor([oracle.e4m3_scale_exp(float(w[c].abs().max())) for c in range(co)], dtype=torch.float64)
        sc = torch.pow(2.0, e).reshape(co, 1, 1, 1, 1)
        out.append((_q8(w / sc) * sc, b))
    return out


def _gpu_codes(pre, det, layer, c_out, rows=None):
    """E4M3 outputs of hidden layer `layer` for the whole batch of det, as
    fp64 [B'][c_out][T][H][H] (B' = the samples in rows, default all)."""
    B, T, H = det.shape[0], pre.T, pre.grid
    out = torch.empty((B, T, H, H, c_out), dtype=torch.uint8, device="cuda")
    pre.activations(torch.from_numpy(np.ascontiguousarray(det).view(np.int64)).cuda(), layer, out)
    torch.cuda.synchronize()
    if rows is not None:
        out = out[torch.as_tensor(rows, device="cuda")]
    return out.cpu().view(torch.float8_e4m3fn).double().permute(0, 4, 1, 2, 3).contiguous()


def _check_layer(name, got, y, eps_abs, act):
    tight.check_stored(name, got, y, eps_abs, act, tight.q_e4m3, say=say)


def _tight_network(pre, det, layers, weights, layout, first, last, rows=None):
    """Every hidden layer's codes, then the logits (of the samples in rows)."""
    d, T = pre.d, pre.T
    sel = det if rows is None else det[rows]
    wq = _layer_weights(weights, layers)
    x = torch.from_numpy(oracle.unpack_paper(d, T, sel, first, last) if layout == "paper"
                         else oracle.unpack(d, T, sel))
    for l in range(len(layers) - 1):
        ci, co, k, act = layers[l]
        w, b = wq[l]
        y = tight.conv(x, w, b)
        eps = (EPS_32 if l == 0 else EPS_MM) * tight.conv_mag(x, w)
        got = _gpu_codes(pre, det, l, co, rows)
        _check_layer("layer %d" % (l + 1), got, y, eps, act)
        x = got
    _, _, logits = run_gpu(pre, det)
    if rows is not None:
        logits = logits[rows]
    w, b = wq[-1]
    k = layers[-1][2]
    ref = tight.conv(x, w, b, k)
    bound = (EPS_MM if k == 3 else EPS_32) * tight.conv_mag(x, w, k=k) + 2.0 ** -22 * ref.abs() + 1e-6
    err = (torch.from_numpy(logits.astype(np.float64)) - ref).abs()
    say("  logits: max err %.3g, max err / bound %.3f" % (float(err.max()), float((err / bound).max())))
    assert bool((err <= bound).all())


TIGHT = [
    dict(name="plaq_3x64_head", layout="plaquette", layers=workload.layer_spec(3, 64), d=5),
    dict(name="plaq_3x128_relu_head", layout="plaquette", layers=workload.layer_spec(3, 128, act=workload.RELU), d=5),
    dict(name="plaq_64_128_64_head", layout="plaquette",
         layers=[(2, 64, 3, 1), (64, 128, 3, 1), (128, 64, 3, 1), (64, 4, 1, 0)], d=7),
    dict(name="paper_m1", layout="paper", layers=workload.paper_model_layers(1), d=7),
    dict(name="paper_256", layout="paper", layers=workload.paper_layer_spec([256, 256, 4], [3, 3, 3]), d=5),
    dict(name="paper_64_d17", layout="paper", layers=workload.paper_layer_spec([64, 64, 4], [3, 3, 3]), d=17),
    # 70 tiles at batch 40: the 128-wide layers as two slices of 64 (batch 1: four of 32)
    dict(name="plaq_4x128_head_d7", layout="plaquette", layers=workload.layer_spec(4, 128), d=7),
]


@pytest.mark.parametrize("batch", [1, 40])
@pytest.mark.parametrize("net", TIGHT, ids=[t["name"] for t in TIGHT])
def test_fp8_layers_tight(cuda, net, batch):
    """Every hidden layer's E4M3 codes from the GPU's own input, then the
    logits from the GPU's last hidden codes (batch 1: split K loops)."""
    layers, layout, d = net["layers"], net["layout"], net["d"]
    T = d
    weights = workload.he_normal_weights(layers, 51 + len(layers))
    det, _ = workload.make_inputs(d, T, batch, 0.02, 0.02, 52)
    first = last = "Z" if layout == "paper" else None
    say("fp8 tight:", net["name"], "batch", batch)
    pre = pdx.Predecoder(weights, d, T, layers, "fp8", max_batch=batch, layout=layout, first=first, last=last)
    _tight_network(pre, det, layers, weights, layout, first, last)
    pre.close()


def test_fp8_layers_tight_full_size(cuda):
    """Workload 3's network (8 x 128, d = 13, T = 13) in fp8 at its full
    batch of 4096, the launch configuration the benchmark times: every
    layer's codes and the logits of three samples (first, middle, last)."""
    d, T, _, layers, weights, det, _ = config_case(3)
    rows = [0, 2048, det.shape[0] - 1]
    say("fp8 tight full size: d", d, "T", T, "B", det.shape[0], "samples", rows)
    pre = pdx.Predecoder(weights, d, T, layers, "fp8", max_batch=det.shape[0])
    _tight_network(pre, det, layers, weights, "plaquette", None, None, rows)
    pre.close()
