"""Residual networks (Model 6, Fig. Model8Representation) on the fp8 path:
E4M3 folded weights with per-channel power-of-two scales, E4M3 activations,
fp32 accumulation, against the oracle's fp8 residual forward, through the C
ABI.  End to end under the fp8 residual bound the oracle derives
(tests/golden/make_resnet_fp8_tolerance.py); per conv under the tight rule of
tight.py: every stored E4M3 code of conv1 and conv2 recomputed in fp64 from
the GPU's own inputs, exact except inside the fp32 summation windows (the fp8
instruction's 2^-16 + 2^-18 of the sum of magnitudes; layer 1's bf16 one),
the fused projections anywhere their own window reaches, and the logits
from the GPU's last block input and intermediate within their bound."""
import json
import os

import numpy as np
import pytest

import oracle
import paper_2604_12841_amd as pdx
import tight
from parity import assert_flips_follow_logits, assert_parity, compare, run_gpu, say
from resnet_cases import RESNET_FP8_CASES, case_inputs
from test_gpu_model6 import _folded

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                                  "resnet_fp8_tolerance.json")))["tol_max_abs_logit_err"]
EPS_MM = 2.0 ** -16 + 2.0 ** -18  # the fp8 instruction's sums
EPS_32 = 2.0 ** -17               # layer 1 (bf16 instruction on the dequantised weights)


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda")


def _scaled_e4m3(w):
    """Per output channel: e4m3(w / 2^e) 2^e with the oracle's scale exponent."""
    out = torch.empty_like(w)
    for o in range(w.shape[0]):
        e = oracle.e4m3_scale_exp(float(w[o].abs().max()))
        out[o] = tight.q_e4m3(w[o] / 2.0 ** e) * 2.0 ** e
    return out


def _pre(case, weights):
    return pdx.Predecoder(weights, case["d"], case["T"], None, "fp8", max_batch=case["B"], layout=case["layout"],
                          first="Z" if case["layout"] == "paper" else None,
                          last="Z" if case["layout"] == "paper" else None, blocks=case["blocks"])


@pytest.mark.parametrize("case", RESNET_FP8_CASES, ids=[c["name"] for c in RESNET_FP8_CASES])
def test_resnet_fp8_parity(cuda, case):
    blocks, d, T, layout = case["blocks"], case["d"], case["T"], case["layout"]
    weights, det, first, last = case_inputs(case)
    say("fp8 resnet", case["name"], "blocks", blocks, "d", d, "T", T, "B", case["B"])
    pre = _pre(case, weights)
    flips, res, logits = run_gpu(pre, det)
    f2, r2, l2 = run_gpu(pre, det)
    pre.close()
    ref = oracle.run_resnet(d, T, det, blocks, weights, bf16=False, layout=layout, first=first, last=last, fp8=True)
    st = compare(d, T, "fp8", *ref, flips, res, logits, layout=layout, tol=TOL)
    say("  stats", st)
    assert_parity(st, "fp8", tol=TOL)
    assert_flips_follow_logits(d, T, det, logits, flips, res, layout)
    assert (flips == f2).all() and (res == r2).all() and (logits == l2).all()


def _codes(pre, ddet, conv, c_out):
    B, T, H = ddet.shape[0], pre.T, pre.grid
    out = torch.empty((B, T, H, H, c_out), dtype=torch.uint8, device="cuda")
    pre.activations(ddet, conv, out)
    torch.cuda.synchronize()
    return out.cpu().view(torch.float8_e4m3fn).double().permute(0, 4, 1, 2, 3).contiguous()


@pytest.mark.parametrize("case", RESNET_FP8_CASES, ids=[c["name"] for c in RESNET_FP8_CASES])
def test_resnet_fp8_convs_tight(cuda, case):
    blocks, d, T, B, layout = case["blocks"], case["d"], case["T"], case["B"], case["layout"]
    weights, det, first, last = case_inputs(case)
    say("fp8 resnet tight", case["name"], "blocks", blocks, "d", d, "T", T, "B", B)
    pre = _pre(case, weights)
    ddet = torch.from_numpy(det.view(np.int64)).cuda()
    x = torch.from_numpy(oracle.unpack_paper(d, T, det, first, last) if layout == "paper"
                         else oracle.unpack(d, T, det))
    x = tight.q_e4m3(x)
    conv = 0
    for k, ((ci, cm, co, act), (w1, b1, w2, b2, wp, bp)) in enumerate(
            zip(blocks, _folded(weights, blocks, quant=_scaled_e4m3))):
        lastb = k == len(blocks) - 1
        # conv1: layer 1 on the bf16 instruction, later ones on the fp8 one
        y = tight.conv(x, w1, b1)
        eps = (EPS_32 if k == 0 else EPS_MM) * tight.conv_mag(x, w1, b1) + tight.U32 * y.abs()
        h = _codes(pre, ddet, conv, cm)
        tight.check_stored("block %d conv1" % (k + 1), h, y, eps, act, tight.q_e4m3, say=say)
        conv += 1
        # the shortcut: the block input, or its projection, fused (first
        # block: an fp32 FMA chain; last block: the fp8 instruction) and
        # rounded to E4M3, so any code its window reaches
        if wp is not None:
            s_exact = tight.conv(x, wp, bp, k=1)
            win = tight.eps_fma_chain(ci) if k == 0 else EPS_MM
            eps_s = win * tight.conv_mag(x, wp, bp, k=1) + tight.U32 * s_exact.abs()
            s_mid, s_lo, s_hi = tight.expected(s_exact, eps_s, tight.NONE, tight.q_e4m3)
            conv += 1
        else:
            s_mid = s_lo = s_hi = x
        y = tight.conv(h, w2, b2) + s_mid
        eps = (EPS_MM * tight.conv_mag(h, w2, b2) + 2 * tight.U32 * (y.abs() + s_mid.abs())
               + torch.maximum(s_hi - s_mid, s_mid - s_lo))
        if not lastb:
            x = _codes(pre, ddet, conv, co)
            tight.check_stored("block %d conv2" % (k + 1), x, y, eps, act, tight.q_e4m3, say=say)
            conv += 1
    flips, res, logits = run_gpu(pre, det)
    pre.close()
    got = torch.from_numpy(logits.astype(np.float64))
    y_lo, y_hi = y - s_mid + s_lo, y - s_mid + s_hi
    bound = EPS_MM * tight.conv_mag(h, w2, b2) + 2.0 ** -22 * (y.abs() + s_mid.abs()) + 1e-6
    err = torch.maximum(y_lo - got, got - y_hi).clamp(min=0.0)
    say("  logits: max err %.3g, max err / bound %.3f" % (float(err.max()), float((err / bound).max())))
    assert bool((err <= bound).all())
    assert_flips_follow_logits(d, T, det, logits, flips, res, layout)
