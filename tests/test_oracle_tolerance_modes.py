"""Pins of the two oracle modes that size parity bounds (test
infrastructure checked like the rest of the oracle):

* the fp32-sum mode of the residual network's conv sums (acc32), which sizes
  the residual networks' end-to-end logit bound: checked bit for bit against
  a numpy float32 sum taken product by product in the same loop order, and
  its fp64 mode against numpy's fp64 sums;
* the fp8 forward with bounded summation errors (fp8_sum_eps, fp8_sum_seed),
  which sizes the fp8 logit bound and excuse band: eps = 0 is the plain fp8
  forward, each sum moves by at most eps * sum|products| and does reach that
  size, both signs occur, and different seeds give different patterns.
The k = 5 forward (Model 3 of Table models) is pinned against PyTorch's
conv3d as the k = 3 one is."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2604_12841_amd import workload
from test_oracle_fp8 import torch_forward_fp8
from test_oracle_forward import torch_forward

NONE, GELU = workload.NONE, workload.GELU_TANH


def _np_conv_sums_f32(x, w, bias):
    """y = fp32 sum over (ci, kt, ki, kj), in that order, of fp32(w x),
    starting from 0, then + bias in fp64 -- written with numpy float32
    arithmetic over shifted views (zero padding)."""
    B, ci, T, H, _ = x.shape
    co, k = w.shape[0], w.shape[2]
    p = (k - 1) // 2
    xp = np.zeros((B, ci, T + 2 * p, H + 2 * p, H + 2 * p))
    xp[:, :, p:p + T, p:p + H, p:p + H] = x
    acc = np.zeros((B, co, T, H, H), dtype=np.float32)
    for c in range(ci):
        for kt in range(k):
            for ki in range(k):
                for kj in range(k):
                    xs = xp[:, c, kt:kt + T, ki:ki + H, kj:kj + H]
                    prod = (w[:, c, kt, ki, kj].reshape(1, co, 1, 1, 1) * xs[:, None]).astype(np.float32)
                    acc = (acc + prod).astype(np.float32)
    return acc.astype(np.float64) + bias.reshape(1, co, 1, 1, 1)


@pytest.mark.parametrize("k", [1, 3])
def test_acc32_is_a_sequential_fp32_sum(k):
    rng = np.random.default_rng(40 + k)
    B, ci, co, T, H = 2, 5, 3, 3, 4
    x = oracle.round_bf16(rng.standard_normal((B, ci, T, H, H)).astype(np.float32)).astype(np.float64)
    w = oracle.round_bf16((rng.standard_normal((co, ci, k, k, k)) * 0.7).astype(np.float32)).astype(np.float64)
    bias = rng.standard_normal(co)
    got32 = oracle.conv_sums(x, w, bias, acc32=True)
    np.testing.assert_array_equal(got32, _np_conv_sums_f32(x, w, bias))
    got64 = oracle.conv_sums(x, w, bias, acc32=False)
    ref64 = F.conv3d(torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(bias), padding=(k - 1) // 2).numpy()
    np.testing.assert_allclose(got64, ref64, rtol=0, atol=1e-12)
    assert (got32 != got64).any()  # the fp32 sums do round


def test_acc32_differs_from_exact_by_at_most_the_fp32_sum_bound():
    """On a 128-channel conv the fp32-sum mode stays within the recursive
    summation bound (n - 1) 2^-24 sum|products| of the fp64 one."""
    rng = np.random.default_rng(44)
    B, ci, co, T, H = 1, 128, 4, 3, 5
    x = rng.standard_normal((B, ci, T, H, H))
    w = rng.standard_normal((co, ci, 3, 3, 3)) * 0.1
    bias = np.zeros(co)
    a = oracle.conv_sums(x, w, bias, acc32=False)
    b = oracle.conv_sums(x, w, bias, acc32=True)
    mag = F.conv3d(torch.from_numpy(np.abs(x)), torch.from_numpy(np.abs(w)), padding=1).numpy()
    n = ci * 27
    assert (np.abs(a - b) <= (n - 1) * 2.0 ** -24 * mag + 1e-12).all()


def _one_layer_case(seed, co=3, ci=6, d=5, T=4, B=2):
    rng = np.random.default_rng(seed)
    layers = [(ci, co, 3, NONE)]
    w = (rng.standard_normal(co * ci * 27) * 0.4).astype(np.float32)
    weights = np.concatenate([w, (rng.standard_normal(co) * 0.3).astype(np.float32)])
    # E4M3 values as inputs, so the fp8 forward's input rounding is exact
    planes = oracle.round_e4m3(rng.standard_normal((B, ci, T, d + 1, d + 1)).astype(np.float32))
    return d, T, layers, weights, planes


def test_fp8_sum_eps_zero_is_the_plain_forward():
    d, T, layers, weights, planes = _one_layer_case(50)
    a = oracle.forward(d, T, planes, layers, weights, False, fp8=True)
    b = oracle.forward(d, T, planes, layers, weights, False, fp8=True, fp8_sum_eps=0.0, fp8_sum_seed=3)
    np.testing.assert_array_equal(a, b)
    # a network with hidden layers too
    layers2 = workload.layer_spec(2, 16)
    w2 = workload.he_normal_weights(layers2, seed=51)
    pl2 = (np.random.default_rng(52).random((2, 2, 4, 6, 6)) < 0.2).astype(np.float64)
    np.testing.assert_array_equal(oracle.forward(5, 4, pl2, layers2, w2, False, fp8=True),
                                  oracle.forward(5, 4, pl2, layers2, w2, False, fp8=True, fp8_sum_eps=0.0))


def test_fp8_sum_eps_moves_each_sum_by_at_most_eps_sum_of_magnitudes():
    """A one-layer network: its logits are fp32(sum + bias), so perturbed minus
    plain is the perturbation itself (up to the two fp32 roundings): within
    eps sum|products|, reaching at least 0.9 of it somewhere, with both
    signs; seeds give different patterns, the same seed the same one."""
    d, T, layers, weights, planes = _one_layer_case(53)
    eps = 2.0 ** -10
    plain = oracle.forward(d, T, planes, layers, weights, False, fp8=True)
    pert = [oracle.forward(d, T, planes, layers, weights, False, fp8=True, fp8_sum_eps=eps, fp8_sum_seed=s)
            for s in (0, 1)]
    # sum|products| from PyTorch's float8 weights (the pinned quantisation)
    ci, co, k, _ = layers[0]
    w = torch.from_numpy(weights[:co * ci * 27].reshape(co, ci, 3, 3, 3).astype(np.float64))
    e = torch.tensor([oracle.e4m3_scale_exp(float(w[c].abs().max())) for c in range(co)], dtype=torch.float64)
    sc = torch.pow(2.0, e).reshape(co, 1, 1, 1, 1)
    wq = (w / sc).float().clamp(-448, 448).to(torch.float8_e4m3fn).double() * sc
    mag = F.conv3d(torch.from_numpy(np.abs(planes)), wq.abs(), padding=1).numpy()
    for p in pert:
        delta = p - plain
        slack = 2.0 ** -23 * (np.abs(plain) + np.abs(p)) + 1e-12
        assert (np.abs(delta) <= eps * mag + slack).all()
        ratio = np.abs(delta) / (eps * mag + 1e-30)
        assert ratio.max() > 0.9
        assert (delta > 0).any() and (delta < 0).any()
    assert (pert[0] != pert[1]).any()
    again = oracle.forward(d, T, planes, layers, weights, False, fp8=True, fp8_sum_eps=eps, fp8_sum_seed=1)
    np.testing.assert_array_equal(again, pert[1])


def test_fp8_sum_eps_requires_fp8():
    d, T, layers, weights, planes = _one_layer_case(54)
    with pytest.raises(ValueError):
        oracle.forward(d, T, planes, layers, weights, True, fp8=False, fp8_sum_eps=1e-3)


@pytest.mark.parametrize("bf16", [False, True])
def test_k5_forward_matches_torch_conv3d(bf16):
    """5 x 5 x 5 kernels (Model 3 of Table models) against conv3d, padding 2."""
    rng = np.random.default_rng(60 + bf16)
    d = T = 5
    layers = workload.paper_layer_spec([8, 8, 4], [5, 5, 5])
    weights = workload.he_normal_weights(layers, seed=61)
    planes = (rng.random((2, 4, T, d, d)) < 0.3).astype(np.float64)
    got = oracle.forward(d, T, planes, layers, weights, bf16=bf16, layout="paper")
    np.testing.assert_allclose(got, torch_forward(planes, layers, weights, bf16), rtol=0,
                               atol=1e-9 if not bf16 else 1e-6)


def test_k5_forward_fp8_matches_torch():
    rng = np.random.default_rng(62)
    d = T = 5
    layers = workload.paper_layer_spec([8, 8, 4], [5, 5, 5])
    weights = workload.he_normal_weights(layers, seed=63)
    planes = (rng.random((1, 4, T, d, d)) < 0.3).astype(np.float64)
    got = oracle.forward(d, T, planes, layers, weights, bf16=False, layout="paper", fp8=True)
    np.testing.assert_allclose(got, torch_forward_fp8(planes, layers, weights), rtol=0, atol=1e-6)


def test_k5_impulse_response_reaches_two_voxels():
    """One 5x5x5 linear layer on an impulse: the response is the flipped
    kernel, nonzero exactly within distance 2 in t, i and j."""
    d, T = 7, 7
    layers = [(4, 1, 5, NONE)]
    w = np.random.default_rng(64).uniform(0.5, 1.0, 4 * 125).astype(np.float32)
    weights = np.concatenate([w, np.zeros(1, np.float32)])
    planes = np.zeros((1, 4, T, d, d))
    planes[0, 2, 3, 3, 3] = 1.0
    y = oracle.forward(d, T, planes, layers, weights, bf16=False, layout="paper")[0, 0]
    nz = np.argwhere(y != 0)
    assert nz.min(axis=0).tolist() == [1, 1, 1] and nz.max(axis=0).tolist() == [5, 5, 5]
    # y[t][i][j] = w[0][2][t - 3 + 2][i - 3 + 2][j - 3 + 2] (cross-correlation)
    wk = w.reshape(1, 4, 5, 5, 5)[0, 2]
    np.testing.assert_allclose(y[1:6, 1:6, 1:6], wk[::-1, ::-1, ::-1], rtol=0, atol=1e-7)
