"""GPU parity of residual networks (Model 6, Sec. VI, Fig.
Model8Representation) against the oracle's residual forward in bf16 mode,
through the C ABI: Model 6 itself on small volumes, projections in a middle
block (widening and narrowing, which also reuse activation buffers at other
row widths), 256-wide slices, ReLU and linear blocks, both layouts, batch 1
(split K loops) and larger batches.  End to end: logits within the bound
that tests/golden/make_resnet_tolerance.py derives from the oracle alone;
flips and residual bits exact outside the sites that bound excuses.  Per
conv: every stored bf16 activation exact outside the fp32-summation window
of tight.py, and the logits within their own sums' bound."""
import json
import os

import numpy as np
import pytest

import oracle
import paper_2604_12841_amd as pdx
import tight
from parity import assert_flips_follow_logits, assert_parity, compare, run_gpu, say
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


# ---- per-conv tight checks ---------------------------------------------
#
# predecoder_activations of a residual network stops after any conv but the
# output layer (per block: conv1, the projection if the block has one,
# conv2) and returns what that conv stored (bf16).  Each conv is recomputed
# in fp64 from the GPU's own inputs -- the folded weights and biases as the
# library uses them (BatchNorm folded in fp64, weights rounded to bf16,
# biases to fp32), the shortcut the GPU stored -- under the rule of tight.py.
# The logits are then checked against the fp64 output conv of the GPU's last
# block input and intermediate, within the bound of their own fp32 sums, and
# the flips and residual against the threshold of the GPU's own logits;
# nothing is excused anywhere.

def _folded(weights, blocks, quant=None):
    """Per block: (w1, b1, w2, b2, wp, bp) as fp64 tensors, BatchNorm folded
    (g = scale / sqrt(var + 1e-5) in fp64, w bf16(fp32(w g)), b fp32((b -
    mean) g + shift)); wp, bp the projection (bf16 weights, fp32 bias) or
    None.  quant: another rounding of the fp32 weights [c_out][...] (the fp8
    path's per-channel scaled E4M3) in place of bf16."""
    quant = quant or tight.q_bf16
    out, off = [], 0

    def take(n):
        nonlocal off
        a = weights[off:off + n].astype(np.float64)
        off += n
        return a

    for ci, cm, co, _act in blocks:
        convs = []
        for cin, cout in ((ci, cm), (cm, co)):
            w = take(cout * cin * 27).reshape(cout, cin, 3, 3, 3)
            b = take(cout)
            scale, shift, mean, var = (take(cout) for _ in range(4))
            g = scale / np.sqrt(var + 1e-5)
            wf = quant(torch.from_numpy((w * g.reshape(-1, 1, 1, 1, 1)).astype(np.float32).astype(np.float64)))
            bf = torch.from_numpy(((b - mean) * g + shift).astype(np.float32).astype(np.float64))
            convs += [wf, bf]
        wp = bp = None
        if ci != co:
            wp = quant(torch.from_numpy(take(co * ci).reshape(co, ci, 1, 1, 1).astype(np.float32).astype(np.float64)))
            bp = torch.from_numpy(take(co).astype(np.float32).astype(np.float64))
        out.append(tuple(convs) + (wp, bp))
    assert off == weights.size
    return out


def _stored(pre, ddet, conv, c_out):
    B, T, H = ddet.shape[0], pre.T, pre.grid
    out = torch.empty((B, T, H, H, c_out), dtype=torch.int16, device="cuda")
    pre.activations(ddet, conv, out)
    torch.cuda.synchronize()
    return tight.bf16_bits_to_double(out.cpu()).permute(0, 4, 1, 2, 3).contiguous()


@pytest.mark.parametrize("case", RESNET_CASES, ids=[c["name"] for c in RESNET_CASES])
def test_resnet_convs_tight(cuda, case):
    blocks, d, T, B, layout = case["blocks"], case["d"], case["T"], case["B"], case["layout"]
    weights, det, first, last = case_inputs(case)
    say("resnet tight", case["name"], "blocks", blocks, "d", d, "T", T, "B", B)
    pre = pdx.Predecoder(weights, d, T, None, "bf16", max_batch=B, layout=layout, first=first, last=last,
                         blocks=blocks)
    ddet = torch.from_numpy(det.view(np.int64)).cuda()
    x = torch.from_numpy(oracle.unpack_paper(d, T, det, first, last) if layout == "paper"
                         else oracle.unpack(d, T, det))
    conv = 0
    for k, ((ci, cm, co, act), (w1, b1, w2, b2, wp, bp)) in enumerate(zip(blocks, _folded(weights, blocks))):
        # conv1: bf16 instructions over 27 c_in products, + bias, activation
        y = tight.conv(x, w1, b1)
        eps = tight.eps_bf16_mfma(27 * ci) * tight.conv_mag(x, w1, b1) + tight.U32 * y.abs()
        h = _stored(pre, ddet, conv, cm)
        tight.check_stored("block %d conv1" % (k + 1), h, y, eps, act, tight.q_bf16, say=say)
        conv += 1
        # shortcut: the block input, or its 1x1x1 projection (an fp32 FMA chain)
        if wp is not None:
            s_exact = tight.conv(x, wp, bp, k=1)
            eps = tight.eps_fma_chain(ci) * tight.conv_mag(x, wp, bp, k=1) + tight.U32 * s_exact.abs()
            s = _stored(pre, ddet, conv, co)
            tight.check_stored("block %d projection" % (k + 1), s, s_exact, eps, tight.NONE, tight.q_bf16, say=say)
            conv += 1
        else:
            s = x
        # conv2 + shortcut: (sum + bias) + shortcut in fp32, then the activation
        y = tight.conv(h, w2, b2) + s
        eps = tight.eps_bf16_mfma(27 * cm) * tight.conv_mag(h, w2, b2) + 2 * tight.U32 * (y.abs() + s.abs())
        if k == len(blocks) - 1 and wp is not None:
            # the output conv computes the last block's projection itself
            # (MFMA sums in another order than the exported one, then bf16):
            # any bf16 value the exact projection's fp32 window reaches
            s_exact = tight.conv(x, wp, bp, k=1)
            eps_s = tight.eps_fma_chain(ci) * tight.conv_mag(x, wp, bp, k=1) + tight.U32 * s_exact.abs()
            _, s_lo, s_hi = tight.expected(s_exact, eps_s, tight.NONE, tight.q_bf16)
            y_lo, y_hi = y - s + s_lo, y - s + s_hi
            eps = eps + 2 * tight.U32 * (s_lo.abs() + s_hi.abs())
        else:
            y_lo = y_hi = y
        if k < len(blocks) - 1:
            x = _stored(pre, ddet, conv, co)
            tight.check_stored("block %d conv2" % (k + 1), x, y, eps, act, tight.q_bf16, say=say)
            conv += 1
    # the output layer: logits of a full run against the GPU's own last inputs
    flips, res, logits = run_gpu(pre, det)
    # the library has no conv after the last one to stop at (past the
    # binding's own range check, through the C ABI)
    import ctypes
    out = torch.empty((B, T, pre.grid, pre.grid, 8), dtype=torch.int16, device="cuda")
    st = pdx.lib().predecoder_activations(pre._h, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream),
                                          ctypes.c_void_p(ddet.data_ptr()), B, conv, ctypes.c_void_p(out.data_ptr()))
    assert st == pdx.PD_ERR_INVALID_ARG
    pre.close()
    got = torch.from_numpy(logits.astype(np.float64))
    err = torch.maximum(y_lo - got, got - y_hi).clamp(min=0.0)  # distance from [y_lo, y_hi]
    bound = eps + 1e-6
    say("  logits: max err %.3g, max err / bound %.3f" % (float(err.max()), float((err / bound).max())))
    assert bool((err <= bound).all())
    assert_flips_follow_logits(d, T, det, logits, flips, res, layout)
