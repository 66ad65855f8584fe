"""The paper's 3x3x3 output layer of four filters (Table models) on its own
kernel (rows = tap x filter, neighbour sums in LDS, units streamed through
the rounds): parity with the oracle across the splits of the grid into
rectangles and of the rounds into ranges, and the logits from the GPU's own
last hidden activations within the fp32 summation bound."""
import numpy as np
import pytest

import oracle
import paper_2604_12841_amd as pdx
from paper_2604_12841_amd import workload
from parity import assert_flips_follow_logits, assert_parity, compare, dev_u64, run_gpu, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda")


# (d, T, B): d 17 / 21 / 25 / 63 split the grid into 2 x 1 ... 7 x 3
# rectangles with rims; small batches split the rounds into one range per
# output round, d = 9 at batch 300 streams each unit through every round
@pytest.mark.parametrize("d,T,B", [(17, 3, 2), (21, 2, 1), (25, 3, 1), (63, 2, 1), (9, 9, 300), (5, 7, 3)])
def test_output_layer_splits(cuda, d, T, B):
    layers = workload.paper_layer_spec([64, 64, 4], [3, 3, 3])
    w = workload.he_normal_weights(layers, seed=700 + d)
    det, _ = workload.make_inputs(d, T, B, 0.01, 0.01, seed=701 + d)
    say("output layer d", d, "T", T, "B", B)
    pre = pdx.Predecoder(w, d, T, layers, "bf16", max_batch=B, layout="paper", first="X", last="Z")
    flips, res, logits = run_gpu(pre, det)
    pre.close()
    ref = oracle.run(d, T, det, layers, w, bf16=True, layout="paper", first="X", last="Z")
    st = compare(d, T, "bf16", ref[0], ref[1], ref[2], flips, res, logits, layout="paper")
    say("  stats", st)
    assert_parity(st, "bf16")


@pytest.mark.parametrize("d,T,B,filters", [(21, 21, 3, [128, 128, 128, 4]), (9, 9, 300, [64, 64, 4]),
                                           (7, 5, 2, [256, 256, 4])])
def test_output_logits_tight(cuda, d, T, B, filters):
    """Logits from the GPU's last hidden activations: exact in fp64 except
    for the fp32 sums (MFMA over the input channels, then the 27 partials
    and the bias), bound (ceil(K/16) + 4) 2^-24 (sum |w x| + |b|) + 2^-24
    |logit|, K = 27 c_in; flips and residual from the GPU's logits."""
    import tight
    layers = workload.paper_layer_spec(filters, [3] * len(filters))
    weights = workload.he_normal_weights(layers, 710 + d)
    det, _ = workload.make_inputs(d, T, B, 0.02, 0.02, 711 + d)
    say("output logits tight d", d, "T", T, "B", B, "filters", filters)
    pre = pdx.Predecoder(weights, d, T, layers, "bf16", max_batch=B, layout="paper", first="Z", last="X")
    ddet = dev_u64(det)
    n = len(layers)
    ci = layers[-1][0]
    out = torch.empty((B, T, d, d, ci), dtype=torch.int16, device="cuda")
    pre.activations(ddet, n - 2, out)
    torch.cuda.synchronize()
    x = tight.bf16_bits_to_double(out.cpu()).permute(0, 4, 1, 2, 3).contiguous()
    off = sum(co * c_in * k ** 3 + co for (c_in, co, k, _) in layers[:-1])
    nw = 4 * ci * 27
    w = tight.q_bf16(torch.from_numpy(weights[off:off + nw].reshape(4, ci, 3, 3, 3).astype(np.float64)))
    b = torch.from_numpy(weights[off + nw:off + nw + 4].astype(np.float64))
    y = tight.conv(x, w, b, 3)
    eps = tight.eps_bf16_mfma(ci * 27) * tight.conv_mag(x, w, b, 3) + tight.U32 * y.abs()
    flips, res, logits = run_gpu(pre, det)
    pre.close()
    err = (torch.from_numpy(logits.astype(np.float64)) - y).abs()
    say("  logits: max err %.3g, max err / bound %.3f" % (float(err.max()), float((err / (eps + 1e-30)).max())))
    assert bool((err <= eps).all())
    assert_flips_follow_logits(d, T, det, logits, flips, res, layout="paper")


def test_output_layer_same_at_any_batch(cuda):
    """A sample's logits do not depend on how the launch splits the rounds
    (one range per output round at batch 1, longer ranges in a batch of 200):
    each output sums the same partials in the same order.  One hidden layer,
    whose activations are bit-identical at any launch size (hidden layers
    after it split their K loops at small batches and round differently)."""
    d = T = 13
    layers = workload.paper_layer_spec([64, 4], [3, 3])
    weights = workload.he_normal_weights(layers, 720)
    B = 200
    det, _ = workload.make_inputs(d, T, B, 0.01, 0.01, 721)
    pre = pdx.Predecoder(weights, d, T, layers, "bf16", max_batch=B, layout="paper", first="Z", last="Z")
    _, _, big = run_gpu(pre, det)
    for s in (0, 99, B - 1):
        _, _, one = run_gpu(pre, det[s:s + 1], batch=1)
        say("sample", s, "batch 1 against batch", B)
        np.testing.assert_array_equal(one[0], big[s])
    pre.close()
