"""Edge cases of the HIP path against the oracle: batches below the handle's
maximum and ragged tails, batch errors, the smallest and largest grids,
extreme detector patterns, the other activations and width changes."""
import numpy as np
import pytest

import oracle
import paper_2604_12841_amd as pdx
from paper_2604_12841_amd import workload
from parity import assert_parity, compare, run_gpu, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda")


def check(d, T, layers, weights, det, dtype, pre=None, batch=None):
    own = pre is None
    if own:
        pre = pdx.Predecoder(weights, d, T, layers, dtype, max_batch=det.shape[0])
    B = det.shape[0] if batch is None else batch
    flips, res, logits = run_gpu(pre, det, batch=B)
    if own:
        pre.close()
    ref = oracle.run(d, T, det[:B], layers, weights, bf16=(dtype == "bf16"))
    st = compare(d, T, dtype, ref[0], ref[1], ref[2], flips, res, logits)
    say("  stats", st)
    assert_parity(st, dtype)
    return flips, res, logits


def test_batches_below_max_and_ragged(cuda):
    d, T = 13, 13
    layers = workload.layer_spec(3, 128)
    w = workload.he_normal_weights(layers, seed=31)
    det, _ = workload.make_inputs(d, T, 32, 0.005, 0.005, seed=32)
    say("batches 1, 7, 32 on one handle with max_batch 32, d 13")
    pre = pdx.Predecoder(w, d, T, layers, "bf16", max_batch=32)
    f1, r1, l1 = check(d, T, layers, w, det, "bf16", pre=pre, batch=1)
    f7, r7, l7 = check(d, T, layers, w, det, "bf16", pre=pre, batch=7)
    f32, r32, l32 = run_gpu(pre, det, batch=32)
    f32b, r32b, l32b = run_gpu(pre, det, batch=32)
    pre.close()
    # a given batch size gives bit-identical results run after run
    np.testing.assert_array_equal(l32, l32b)
    np.testing.assert_array_equal(f32, f32b)
    np.testing.assert_array_equal(r32, r32b)
    # batch sizes that split the K loops differently sum in another order (and
    # a bf16 activation can round the other way): they agree under the
    # parity rule
    for other in (l7[0], l32[0]):
        np.testing.assert_allclose(other, l1[0], rtol=0, atol=2e-2)
    st = compare(d, T, "bf16", l32[:7].astype(np.float64), f32[:7], r32[:7], f7, r7, l7)
    say("  batch 7 against batch 32", st)
    assert_parity(st, "bf16")


def test_batch_errors(cuda):
    d, T = 5, 5
    layers = workload.layer_spec(2, 64)
    w = workload.he_normal_weights(layers, seed=3)
    det, _ = workload.make_inputs(d, T, 4, 0.01, 0.01, seed=4)
    pre = pdx.Predecoder(w, d, T, layers, "bf16", max_batch=2)
    ddet = torch.from_numpy(det.view(np.int64)).cuda()
    flips = torch.zeros((4, pre.flip_words), dtype=torch.int64, device="cuda")
    res = torch.zeros((4, pre.det_words), dtype=torch.int64, device="cuda")
    # batches the library itself rejects (the binding checks only buffer sizes
    # and batch >= 1): through the C ABI directly, then through the binding
    import ctypes
    for bad in (0, 3, -1):
        st = pdx.lib().predecoder_run(pre._h, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream),
                                      ctypes.c_void_p(ddet.data_ptr()), bad, ctypes.c_void_p(flips.data_ptr()),
                                      ctypes.c_void_p(res.data_ptr()), None)
        assert st == pdx.PD_ERR_INVALID_ARG
    with pytest.raises(pdx.PredecoderError) as e:
        pre.run(ddet, flips, res, batch=3)
    assert e.value.status == pdx.PD_ERR_INVALID_ARG
    for bad in (0, -1):
        with pytest.raises(ValueError):
            pre.run(ddet, flips, res, batch=bad)
    # the handle stays usable after an error
    check(d, T, layers, w, det[:2], "bf16", pre=pre)
    pre.close()


@pytest.mark.parametrize("d,T,B", [(3, 1, 5), (3, 2, 1), (5, 1, 3), (11, 40, 2), (63, 3, 1)])
def test_grid_extremes(cuda, d, T, B):
    layers = workload.layer_spec(2, 64)
    w = workload.he_normal_weights(layers, seed=100 + d)
    det, _ = workload.make_inputs(d, T, B, 0.01, 0.01, seed=200 + T)
    say("grid d", d, "T", T, "B", B)
    check(d, T, layers, w, det, "bf16")


@pytest.mark.parametrize("pattern", ["zeros", "ones"])
def test_extreme_detectors(cuda, pattern):
    d, T, B = 9, 9, 3
    layers = workload.layer_spec(3, 64)
    w = workload.he_normal_weights(layers, seed=41)
    W = pdx.det_words(d, T)
    # all-ones also sets the padding bits, which the path must ignore
    det = np.zeros((B, W), np.uint64) if pattern == "zeros" else np.full((B, W), np.uint64(2**64 - 1))
    say("detectors all", pattern)
    check(d, T, layers, w, det, "bf16")


@pytest.mark.parametrize("act", [pdx.ACT_RELU, pdx.ACT_NONE])
@pytest.mark.parametrize("dtype,width", [("bf16", 64), ("bf16", 128), ("fp32", 32)])
def test_other_activations(cuda, act, dtype, width):
    d, T, B = 7, 5, 3
    layers = workload.layer_spec(3, width, act=act)
    w = workload.he_normal_weights(layers, seed=51)
    det, _ = workload.make_inputs(d, T, B, 0.02, 0.02, seed=52)
    say("activation", act, dtype, "width", width)
    check(d, T, layers, w, det, dtype)


def test_width_changes(cuda):
    d, T, B = 9, 7, 2
    layers = [(2, 64, 3, pdx.ACT_GELU_TANH), (64, 128, 3, pdx.ACT_GELU_TANH), (128, 64, 3, pdx.ACT_GELU_TANH),
              (64, 128, 3, pdx.ACT_GELU_TANH), (128, 4, 1, pdx.ACT_NONE)]
    w = workload.he_normal_weights(layers, seed=61)
    det, _ = workload.make_inputs(d, T, B, 0.01, 0.01, seed=62)
    say("width changes 2-64-128-64-128-4")
    check(d, T, layers, w, det, "bf16")


@pytest.mark.parametrize("width,d,T,B", [(64, 9, 7, 3), (128, 13, 5, 2), (128, 25, 3, 1), (64, 31, 2, 1)])
def test_single_hidden_layer(cuda, width, d, T, B):
    # layer 1 carries the head and the threshold (flat and box tilings)
    layers = workload.layer_spec(1, width)
    w = workload.he_normal_weights(layers, seed=71 + d)
    det, _ = workload.make_inputs(d, T, B, 0.01, 0.01, seed=72 + d)
    say("one hidden layer, width", width, "d", d, "T", T, "B", B)
    check(d, T, layers, w, det, "bf16")


def test_buffer_reuse_at_other_row_widths(cuda):
    """Widths that alternate unevenly over the two activation buffers (64,
    128, 128, 64: each buffer is written at one width and later at another):
    the zero halo the 3x3x3 layers read must stay zero."""
    d, T = 5, 4
    G = workload.GELU_TANH
    layers = [(2, 64, 3, G), (64, 128, 3, G), (128, 128, 3, G), (128, 64, 3, G), (64, 4, 1, workload.NONE)]
    weights = workload.he_normal_weights(layers, 91)
    det, _ = workload.make_inputs(d, T, 3, 0.02, 0.02, 92)
    pre = pdx.Predecoder(weights, d, T, layers, "bf16", max_batch=3)
    flips, res, logits = run_gpu(pre, det)
    f2, r2, l2 = run_gpu(pre, det)
    pre.close()
    st = compare(d, T, "bf16", *oracle.run(d, T, det, layers, weights, bf16=True), flips, res, logits)
    say("  reuse at other widths bf16", st)
    assert_parity(st, "bf16")
    assert (logits == l2).all()
    # the fp32 path (its own kernels and widths)
    lf = [(2, 16, 3, G), (16, 32, 3, G), (32, 64, 3, G), (64, 16, 3, G), (16, 4, 1, workload.NONE)]
    wf = workload.he_normal_weights(lf, 93)
    pre = pdx.Predecoder(wf, d, T, lf, "fp32", max_batch=3)
    flips, res, logits = run_gpu(pre, det)
    pre.close()
    st = compare(d, T, "fp32", *oracle.run(d, T, det, lf, wf, bf16=False), flips, res, logits)
    say("  reuse at other widths fp32", st)
    assert_parity(st, "fp32")


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_layer1_same_at_any_launch_size(cuda, dtype):
    """Layer 1 divides its work by launch size (two 32-voxel blocks per wave
    on large launches; one block, and for 128 channels its two 64-channel
    halves on two waves, on small ones): a sample's layer-1 activations are
    bit-identical either way (no split sums in layer 1)."""
    d = T = 5
    layers = workload.layer_spec(3, 128)
    weights = workload.he_normal_weights(layers, 81)
    B = 800  # 800 x 180 voxels: past the large-launch threshold
    det, _ = workload.make_inputs(d, T, B, 0.01, 0.01, 82)
    pre = pdx.Predecoder(weights, d, T, layers, dtype, max_batch=B)
    ddet = torch.from_numpy(np.ascontiguousarray(det).view(np.int64)).cuda()
    H = pre.grid
    el = torch.uint8 if dtype == "fp8" else torch.int16
    big = torch.empty((B, T, H, H, 128), dtype=el, device="cuda")
    pre.activations(ddet, 0, big)
    one = torch.empty((1, T, H, H, 128), dtype=el, device="cuda")
    for s in (0, 517, B - 1):
        say("layer 1", dtype, "sample", s)
        pre.activations(ddet[s:s + 1], 0, one, batch=1)
        torch.cuda.synchronize()
        assert torch.equal(one[0].cpu(), big[s].cpu())
    pre.close()


@pytest.mark.parametrize("width,n,B", [(64, 6, 1), (64, 6, 40), (128, 4, 1), (128, 4, 20), (128, 4, 40)])
def test_sliced_layers_tight(cuda, width, n, B):
    """n hidden layers of 64 or 128 channels at d = T = 9 (4, 70 and 141
    tiles at batches 1, 20 and 40): at batch 1 each C -> C layer runs as
    32-channel output slices (the last, which carries the head, where whole
    it would split its K loops: the 128-wide one, its slices' sums then
    finished with the head by the second kernel), at batch 20 a 128-wide one
    but the last as two slices of 64, at batch 40 whole.  Either way every
    hidden layer's stored bf16 activations are checked from the GPU's own
    input under the rule of tests/tight.py, then the logits from the GPU's
    last hidden activations within their own sums' bound."""
    import tight
    from parity import dev_u64
    d = T = 9
    H = d + 1
    layers = workload.layer_spec(n, width)
    weights = workload.he_normal_weights(layers, 81 + width)
    det, _ = workload.make_inputs(d, T, B, 0.02, 0.02, 82)
    say("%d x %d layers, tight, d = T =" % (n, width), d, "batch", B)
    pre = pdx.Predecoder(weights, d, T, layers, "bf16", max_batch=B)
    ddet = dev_u64(det)
    x = torch.from_numpy(oracle.unpack(d, T, det))
    off = 0
    for l, (ci, co, k, act) in enumerate(layers):
        nw = co * ci * k ** 3
        w = tight.q_bf16(torch.from_numpy(weights[off:off + nw].reshape(co, ci, k, k, k).astype(np.float64)))
        b = torch.from_numpy(weights[off + nw:off + nw + co].astype(np.float64))
        off += nw + co
        y = tight.conv(x, w, b, k)
        # the 1x1x1 head sums on the vector ALU: an fp32 chain's bound
        e = tight.eps_bf16_mfma(ci * k ** 3) if k > 1 else tight.eps_fma_chain(ci)
        eps = e * tight.conv_mag(x, w, b, k) + tight.U32 * y.abs()
        if l < len(layers) - 1:
            out = torch.empty((B, T, H, H, co), dtype=torch.int16, device="cuda")
            pre.activations(ddet, l, out)
            torch.cuda.synchronize()
            got = tight.bf16_bits_to_double(out.cpu()).permute(0, 4, 1, 2, 3).contiguous()
            tight.check_stored("layer %d" % (l + 1), got, y, eps, act, tight.q_bf16, say=say)
            x = got
    _, _, logits = run_gpu(pre, det)
    pre.close()
    err = (torch.from_numpy(logits.astype(np.float64)) - y).abs()
    say("  logits: max err %.3g, max err / bound %.3f" % (float(err.max()), float((err / (eps + 1e-6)).max())))
    assert bool((err <= eps + 1e-6).all())
