"""Pins of the oracle's fp8 mode (the paper deploys its models in FP8,
Sec. VI; OCP E4M3 with the scaling reading stated in oracle.c): the E4M3
codes against PyTorch's float8_e4m3fn, saturation, the weight scale rule,
and the whole fp8 forward against a PyTorch conv3d pipeline that applies the
same quantisation points with PyTorch's own fp8 conversion."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2604_12841_amd import workload

GELU, NONE, RELU = workload.GELU_TANH, workload.NONE, workload.RELU


def torch_codes(x):
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def torch_values():
    return torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).double().numpy()


def test_e4m3_values_match_torch():
    ref = torch_values()
    got = np.array([oracle.e4m3_value(c) for c in range(256)])
    nan = np.isnan(ref)
    assert list(np.flatnonzero(nan)) == [0x7F, 0xFF]
    assert np.isnan(got[nan]).all()
    np.testing.assert_array_equal(got[~nan], ref[~nan])
    # closed forms of the format: largest finite, smallest normal and subnormal
    assert got[0x7E] == 448.0 and got[0x08] == 2.0 ** -6 and got[0x01] == 2.0 ** -9


def test_e4m3_rounding_matches_torch_in_range():
    rng = np.random.default_rng(8)
    vals = torch_values()[:0x7F]  # non-negative finite, increasing
    mids = (vals[:-1] + vals[1:]) / 2  # exact ties, both parities of the lower code
    x = np.concatenate([
        rng.standard_normal(3000) * 4,
        rng.standard_normal(1000) * 2.0 ** -8,  # subnormal range
        rng.uniform(-464, 464, 1000),
        mids, -mids,
        np.nextafter(mids.astype(np.float32), np.float32(0)),
        np.nextafter(mids.astype(np.float32), np.float32(1e9)),
        [0.0, -0.0, 448.0, -448.0, 460.0, 464.0],
    ]).astype(np.float32)
    np.testing.assert_array_equal(oracle.e4m3_code(x), torch_codes(x))
    np.testing.assert_array_equal(oracle.round_e4m3(x), torch.from_numpy(x).to(torch.float8_e4m3fn).double().numpy())


def test_e4m3_saturation_and_nan():
    x = np.array([465.0, 500.0, 1e6, 3e38, np.inf, -470.0, -np.inf], np.float32)
    assert list(oracle.e4m3_code(x)) == [0x7E] * 5 + [0xFE] * 2
    assert oracle.e4m3_code(np.array([np.nan], np.float32))[0] == 0x7F


def test_scale_exponent_rule():
    rng = np.random.default_rng(9)
    amax = np.concatenate([np.exp(rng.uniform(-40, 40, 2000)), [448.0, 449.0, 224.0, 896.0, 1e-30]])
    for a in amax:
        e = oracle.e4m3_scale_exp(a)
        assert math.ldexp(a, -e) <= 448.0 < math.ldexp(a, -(e - 1)), (a, e)
    assert oracle.e4m3_scale_exp(448.0) == 0 and oracle.e4m3_scale_exp(449.0) == 1
    assert oracle.e4m3_scale_exp(224.0) == -1 and oracle.e4m3_scale_exp(0.0) == 0


def torch_forward_fp8(planes, layers, weights):
    """conv3d pipeline with PyTorch's float8_e4m3fn conversions: weights
    e4m3(w / 2^e) * 2^e per output channel, conv inputs e4m3 (saturated at
    448), pre-activation fp32, activation in fp64 then fp32, logits fp32."""
    def q(t):
        return t.float().clamp(-448.0, 448.0).to(torch.float8_e4m3fn).double()

    x = q(torch.from_numpy(planes))
    off = 0
    for li, (ci, co, k, act) in enumerate(layers):
        nw = co * ci * k ** 3
        w = torch.from_numpy(weights[off:off + nw].reshape(co, ci, k, k, k).astype(np.float64))
        b = torch.from_numpy(weights[off + nw:off + nw + co].astype(np.float64))
        off += nw + co
        e = torch.tensor([oracle.e4m3_scale_exp(float(w[c].abs().max())) for c in range(co)], dtype=torch.float64)
        scale = torch.pow(2.0, e).reshape(co, 1, 1, 1, 1)
        wq = q(w / scale) * scale
        y = F.conv3d(x, wq, b, padding=(k - 1) // 2).float().double()
        if li < len(layers) - 1:
            if act == GELU:
                y = F.gelu(y, approximate="tanh")
            elif act == RELU:
                y = F.relu(y)
            y = q(y)
        x = y
    return x.numpy()


@pytest.mark.parametrize("d,T,n_hidden,width,B,act", [
    (5, 5, 4, 32, 2, GELU),
    (9, 3, 3, 64, 1, GELU),
    (3, 1, 3, 8, 3, GELU),
    (7, 4, 2, 16, 2, RELU),
])
def test_forward_fp8_matches_torch(d, T, n_hidden, width, B, act):
    rng = np.random.default_rng(d * 100 + T)
    layers = workload.layer_spec(n_hidden, width, act=act)
    weights = workload.he_normal_weights(layers, seed=d + 7)
    planes = (rng.random((B, 2, T, d + 1, d + 1)) < 0.1).astype(np.float64)
    got = oracle.forward(d, T, planes, layers, weights, bf16=False, fp8=True)
    ref = torch_forward_fp8(planes, layers, weights)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-6)


def test_forward_fp8_paper_layout_matches_torch():
    d = T = 5
    layers = workload.paper_layer_spec([16, 16, 4], [3, 3, 3])
    weights = workload.he_normal_weights(layers, seed=11)
    det, _ = workload.make_inputs(d, T, 2, 0.05, 0.05, 12)
    planes = oracle.unpack_paper(d, T, det, "Z", "Z")
    got = oracle.forward(d, T, planes, layers, weights, bf16=False, layout="paper", fp8=True)
    np.testing.assert_allclose(got, torch_forward_fp8(planes, layers, weights), rtol=0, atol=1e-6)


def test_fp8_weights_within_half_a_step_of_exact():
    """The fp8 weights of a one-layer linear network are each within half an
    E4M3 step of the fp32 weights: on an impulse input the output is the
    flipped kernel, so |y_fp8 - y_exact| <= 2^-4 |w| + 2^-10 2^e per tap."""
    rng = np.random.default_rng(13)
    co, ci = 3, 2
    w = (rng.standard_normal(co * ci * 27) * 0.3).astype(np.float32)
    weights = np.concatenate([w, np.zeros(co, np.float32)])
    planes = np.zeros((1, ci, 3, 3, 3))
    planes[0, 0, 1, 1, 1] = 1.0
    layers = [(ci, co, 3, NONE)]
    y8 = oracle.forward(2, 3, planes, layers, weights, bf16=False, fp8=True)[0]
    y = oracle.forward(2, 3, planes, layers, weights, bf16=False)[0]
    wr = w.reshape(co, ci, 27)
    for c in range(co):
        e = oracle.e4m3_scale_exp(np.abs(wr[c]).max())
        bound = np.abs(y[c]) * 2.0 ** -4 + 2.0 ** (e - 10)
        assert (np.abs(y8[c] - y[c]) <= bound + 1e-12).all()
        assert (y8[c] != y[c]).any()  # the rounding did act
