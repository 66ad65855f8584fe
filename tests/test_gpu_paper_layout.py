"""The paper's own layout on the GPU against the oracle (Sec. IV.B.1, Table
models): four input channels on the D x D data-qubit grid with the geometric
channels cleared in the preparation / measurement rounds, a 4-channel first
layer, and a 3x3x3 output layer of four filters (or a 1x1x1 head)."""
import numpy as np
import pytest

import oracle
import paper_2604_12841_amd as pdx
from paper_2604_12841_amd import workload
from parity import assert_parity, compare, dev_u64, run_gpu, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda")


def check(d, T, B, layers, seed, first="Z", last="Z", p=0.01):
    w = workload.he_normal_weights(layers, seed=seed)
    det, _ = workload.make_inputs(d, T, B, p, p, seed=seed + 1)
    say("paper layout d", d, "T", T, "B", B, "layers", layers, "first", first, "last", last)
    pre = pdx.Predecoder(w, d, T, layers, "bf16", max_batch=B, layout="paper", first=first, last=last)
    flips, res, logits = run_gpu(pre, det)
    pre.close()
    ref = oracle.run(d, T, det, layers, w, bf16=True, layout="paper", first=first, last=last)
    st = compare(d, T, "bf16", ref[0], ref[1], ref[2], flips, res, logits, layout="paper")
    say("  stats", st)
    assert_parity(st, "bf16")


@pytest.mark.parametrize("d,T,B,filters", [
    (5, 5, 3, [64, 64, 4]),
    (7, 7, 2, [128, 128, 128, 4]),        # Model 1's layer list
    (9, 5, 2, [128] * 5 + [4]),           # Model 4's layer list
    (13, 13, 2, [128, 128, 128, 4]),      # Model 1 at 13^3
    (3, 1, 4, [64, 4]),                   # one hidden layer, a single round
])
def test_paper_models_3x3x3_output(cuda, d, T, B, filters):
    check(d, T, B, workload.paper_layer_spec(filters, [3] * len(filters)), seed=300 + d)


@pytest.mark.parametrize("d,T,B,filters", [
    (5, 3, 2, [256, 256, 4]),              # Model 2's widths
    (5, 3, 1, [256] * 5 + [4]),           # Model 5's layer list
    (7, 4, 2, [128, 256, 128, 4]),         # 128 -> 256 -> 128 slices
    (9, 3, 1, [256, 64, 4]),               # 256 -> 64
])
def test_width_256_as_two_slices(cuda, d, T, B, filters):
    check(d, T, B, workload.paper_layer_spec(filters, [3] * len(filters)), seed=380 + d + len(filters))


def test_paper_model_on_box_tiles(cuda):
    # d = 31 gives box tiles (the 31 x 31 grid is too wide for flat ones)
    check(31, 3, 1, workload.paper_layer_spec([64, 64, 4], [3, 3, 3]), seed=331)


@pytest.mark.parametrize("first,last", [(None, None), ("X", "X"), ("Z", "X"), ("X", None)])
def test_boundary_bases(cuda, first, last):
    check(5, 4, 2, workload.paper_layer_spec([64, 64, 4], [3, 3, 3]), seed=340, first=first, last=last)


@pytest.mark.parametrize("filters", [[64, 64, 4], [128, 4]])
def test_paper_layout_with_1x1x1_head(cuda, filters):
    kernels = [3] * (len(filters) - 1) + [1]
    check(7, 5, 3, workload.paper_layer_spec(filters, kernels), seed=350 + len(filters))


def test_paper_unpack_planes_exact(cuda):
    d, T, B = 7, 4, 3
    layers = workload.paper_layer_spec([64, 4], [3, 3])
    w = workload.he_normal_weights(layers, seed=360)
    det, _ = workload.make_inputs(d, T, B, 0.05, 0.05, seed=361)
    pre = pdx.Predecoder(w, d, T, layers, "bf16", max_batch=B, layout="paper", first="X", last="Z")
    planes = torch.full((B, T, d, d, 4), -1, dtype=torch.int16, device="cuda")
    pre.unpack(dev_u64(det), planes)
    torch.cuda.synchronize()
    pre.close()
    got = planes.cpu().view(torch.bfloat16).float().numpy()
    ref = oracle.unpack_paper(d, T, det, "X", "Z").transpose(0, 2, 3, 4, 1)
    np.testing.assert_array_equal(got, ref)


def test_paper_layout_fp32_is_unsupported(cuda):
    layers = workload.paper_layer_spec([64, 4], [3, 3])
    w = workload.he_normal_weights(layers, seed=370)
    with pytest.raises(pdx.PredecoderError) as e:
        pdx.Predecoder(w, 5, 3, layers, "fp32", max_batch=1, layout="paper")
    assert e.value.status == pdx.PD_ERR_UNSUPPORTED


# ---- 5x5x5 kernels (Model 3 of Table models) -----------------------------

@pytest.mark.parametrize("d,T,B,filters", [
    (5, 5, 2, [64, 64, 4]),                # the smallest 5x5x5 network, a halo of two
    (7, 6, 3, [128, 128, 4]),
    (9, 4, 1, [64, 64, 64, 4]),             # three 64-wide 5x5x5 layers
    (13, 13, 1, [128, 128, 128, 4]),        # Model 3 at 13^3, batch 1 (split K loops)
    (13, 13, 2, [128, 128, 128, 4]),        # ... batch 2
    (31, 2, 1, [64, 64, 4]),                # box tiles across a 31 x 31 grid
])
def test_paper_models_5x5x5(cuda, d, T, B, filters):
    check(d, T, B, workload.paper_layer_spec(filters, [5] * len(filters)), seed=500 + d + len(filters))


def test_5x5x5_layers_tight(cuda):
    """Model 3's layer list at d = 7, batch 2: every layer's stored bf16
    activations from the GPU's own input under the rule of tests/tight.py
    (bf16 matrix instructions over 125 taps x c_in products), then the
    logits from the GPU's last hidden activations within their own sums'
    bound, and the flips and residual from the GPU's logits."""
    import tight
    from parity import assert_flips_follow_logits
    d = T = 7
    B = 2
    layers = workload.paper_model_layers(3)
    weights = workload.he_normal_weights(layers, 4003)
    det, _ = workload.make_inputs(d, T, B, 0.02, 0.02, 5007)
    pre = pdx.Predecoder(weights, d, T, layers, "bf16", max_batch=B, layout="paper", first="Z", last="Z")
    ddet = dev_u64(det)
    x = torch.from_numpy(oracle.unpack_paper(d, T, det, "Z", "Z"))
    off = 0
    for l, (ci, co, k, act) in enumerate(layers):
        nw = co * ci * k ** 3
        w = tight.q_bf16(torch.from_numpy(weights[off:off + nw].reshape(co, ci, k, k, k).astype(np.float64)))
        b = torch.from_numpy(weights[off + nw:off + nw + co].astype(np.float64))
        off += nw + co
        y = tight.conv(x, w, b, k)
        eps = tight.eps_bf16_mfma(ci * k ** 3) * tight.conv_mag(x, w, b, k) + tight.U32 * y.abs()
        if l < len(layers) - 1:
            out = torch.empty((B, T, d, d, co), dtype=torch.int16, device="cuda")
            pre.activations(ddet, l, out)
            torch.cuda.synchronize()
            got = tight.bf16_bits_to_double(out.cpu()).permute(0, 4, 1, 2, 3).contiguous()
            tight.check_stored("layer %d (5x5x5)" % (l + 1), got, y, eps, act, tight.q_bf16, say=say)
            x = got
    flips, res, logits = run_gpu(pre, det)
    pre.close()
    err = (torch.from_numpy(logits.astype(np.float64)) - y).abs()
    say("  logits: max err %.3g, max err / bound %.3f" % (float(err.max()), float((err / (eps + 1e-6)).max())))
    assert bool((err <= eps + 1e-6).all())
    assert_flips_follow_logits(d, T, det, logits, flips, res, layout="paper")


def test_5x5x5_layer1_same_at_any_launch_size(cuda):
    """The 5x5x5 first layer gives each wave up to eight 32-voxel blocks on
    large launches and one on small ones, one 64-channel half per workgroup
    either way: a sample's layer-1 activations are bit-identical at batch 1
    and inside a batch of 240 (eight blocks per wave at d = 13)."""
    d = T = 13
    B = 240
    layers = workload.paper_model_layers(3)
    weights = workload.he_normal_weights(layers, 4003)
    det, _ = workload.make_inputs(d, T, B, 0.01, 0.01, 5013)
    pre = pdx.Predecoder(weights, d, T, layers, "bf16", max_batch=B, layout="paper", first="Z", last="Z")
    ddet = dev_u64(det)
    big = torch.empty((B, T, d, d, 128), dtype=torch.int16, device="cuda")
    pre.activations(ddet, 0, big)
    one = torch.empty((1, T, d, d, 128), dtype=torch.int16, device="cuda")
    for s in (0, 117, B - 1):
        say("5x5x5 layer 1 sample", s)
        pre.activations(ddet[s:s + 1], 0, one, batch=1)
        torch.cuda.synchronize()
        assert torch.equal(one[0].cpu(), big[s].cpu())
    pre.close()
