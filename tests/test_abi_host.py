"""Host-side checks of the C ABI (no kernel launches): the library loads and
exports every function declared in include/predecoder.h, the size helpers and
the parameter-count rule agree with the paper's tables, and create() rejects
misuse before touching the device."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2604_12841_amd as pdx
from conftest import ROOT, gpu_available
from paper_2604_12841_amd import workload

HEADER = os.path.join(ROOT, "include", "predecoder.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(predecoder_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 10
    L = pdx.lib()
    for n in names:
        assert hasattr(L, n), n
    assert sorted(pdx.EXPORTS) == names


def test_word_counts():
    for d, T in [(3, 1), (5, 5), (9, 9), (13, 13), (25, 25), (31, 31)]:
        assert pdx.det_words(d, T) == -(-T * (d * d - 1) // 64)
        assert pdx.flip_words(d, T) == -(-T * (3 * d * d - 1) // 64)
    assert pdx.det_words(13, 13) == 35 and pdx.flip_words(13, 13) == 103
    assert pdx.det_words(0, 5) == -1 and pdx.flip_words(5, 0) == -1


def test_weight_count_matches_paper_tables(golden_dir):
    for line in open(os.path.join(golden_dir, "param_counts.txt")):
        if line.startswith("#") or not line.strip():
            continue
        m, filt, ks, printed = line.split()
        layers, ci = [], 4
        for f, k in zip(filt.split(","), ks.split(",")):
            layers.append((ci, int(f), int(k), 1))
            ci = int(f)
        n = pdx.weight_count(layers)
        assert n == (912772 if m == "1" else int(printed))
    # Model 6: conv layers of the residual network (BatchNorm adds 2 per channel)
    convs, bn = [], 0
    lines = [l.split() for l in open(os.path.join(golden_dir, "model6.txt")) if l.strip() and not l.startswith("#")]
    printed = int(lines[0][0])
    for p in lines[1:]:
        if p[0] == "conv":
            convs.append((int(p[1]), int(p[2]), int(p[3]), 1))
        else:
            bn += 2 * int(p[1])
    assert sum(pdx.weight_count([c]) for c in convs) + bn == printed
    assert pdx.weight_count([]) == 0


def test_workload_weight_sizes():
    for cfg in workload.CONFIGS:
        layers = workload.config_layers(cfg)
        assert workload.config_weights(cfg).size == pdx.weight_count(layers)


def test_status_strings():
    for s in range(5):
        assert pdx.status_string(s)
    assert "invalid" in pdx.status_string(pdx.PD_ERR_INVALID_ARG)


def _create(weights, d, T, layers, dtype=pdx.DTYPE_BF16, max_batch=4, n_weights=None, out=True):
    L = pdx.lib()
    w = np.ascontiguousarray(weights, dtype=np.float32)
    arr = pdx._layers(layers) if layers is not None else None
    h = ctypes.c_void_p()
    st = L.predecoder_create(w.ctypes.data_as(ctypes.c_void_p) if w.size else None,
                             w.size if n_weights is None else n_weights, d, T, arr,
                             len(layers) if layers else 0, dtype, max_batch, ctypes.byref(h) if out else None)
    if st == pdx.PD_OK:
        L.predecoder_destroy(h)
    return st


LAYERS = workload.layer_spec(2, 64)
W = workload.he_normal_weights(LAYERS, 0)


@pytest.mark.parametrize("case", [
    dict(d=4), dict(d=1), dict(d=-3), dict(T=0), dict(dtype=7), dict(max_batch=0),
    dict(layers=[(3, 64, 3, 1), (64, 64, 3, 1), (64, 4, 1, 0)]),   # first c_in must be 2
    dict(layers=[(2, 64, 3, 1), (64, 64, 3, 1), (64, 5, 1, 0)]),   # head must give 4 channels
    dict(layers=[(2, 64, 3, 1), (32, 64, 3, 1), (64, 4, 1, 0)]),   # broken chain
    dict(layers=[(2, 64, 4, 1), (64, 64, 3, 1), (64, 4, 1, 0)]),   # even kernel
    dict(layers=[(2, 64, 3, 1), (64, 64, 3, 1), (64, 4, 1, 1)]),   # activated head
    dict(layers=[(2, 64, 3, 9), (64, 64, 3, 1), (64, 4, 1, 0)]),   # unknown activation
    dict(n_weights=W.size - 1),
    dict(out=False),
])
def test_create_rejects_misuse(case):
    args = dict(weights=W, d=5, T=3, layers=LAYERS)
    args.update(case)
    assert _create(**args) == pdx.PD_ERR_INVALID_ARG


def test_create_rejects_null_pointers():
    L = pdx.lib()
    h = ctypes.c_void_p()
    arr = pdx._layers(LAYERS)
    assert L.predecoder_create(None, W.size, 5, 3, arr, len(LAYERS), 1, 4, ctypes.byref(h)) == pdx.PD_ERR_INVALID_ARG
    w = np.ascontiguousarray(W)
    assert L.predecoder_create(w.ctypes.data_as(ctypes.c_void_p), W.size, 5, 3, None, 3, 1, 4,
                               ctypes.byref(h)) == pdx.PD_ERR_INVALID_ARG
    assert h.value is None


@pytest.mark.parametrize("layers,dtype", [
    ([(2, 64, 5, 1), (64, 4, 1, 0)], pdx.DTYPE_BF16),          # 5x5x5 hidden layer
    ([(2, 96, 3, 1), (96, 4, 1, 0)], pdx.DTYPE_BF16),          # width 96 on the bf16 path
    ([(2, 64, 3, 1), (64, 4, 3, 0)], pdx.DTYPE_BF16),          # 3x3x3 head
    ([(2, 4, 1, 0)], pdx.DTYPE_BF16),                          # no hidden layer
    ([(2, 20, 3, 1), (20, 4, 1, 0)], pdx.DTYPE_FP32),          # fp32 width not a multiple of 8
    ([(2, 64, 3, 1), (64, 4, 1, 0)], pdx.DTYPE_FP8),           # fp8: one hidden layer with a 1x1x1 head
    ([(2, 32, 3, 1), (32, 32, 3, 1), (32, 4, 1, 0)], pdx.DTYPE_FP8),  # fp8 width 32
])
def test_create_unsupported_shapes(layers, dtype):
    w = workload.he_normal_weights(layers, 0)
    assert _create(w, 5, 3, layers, dtype=dtype) == pdx.PD_ERR_UNSUPPORTED


def test_create_unsupported_distance():
    assert _create(W, 65, 3, LAYERS) == pdx.PD_ERR_UNSUPPORTED
    assert _create(W, 5, 1024, LAYERS) == pdx.PD_ERR_UNSUPPORTED


@pytest.mark.skipif(gpu_available(), reason="checks the no-device error path")
def test_create_without_device_reports_device_error():
    assert _create(W, 5, 3, LAYERS) == pdx.PD_ERR_DEVICE


def test_run_rejects_null_handle():
    L = pdx.lib()
    assert L.predecoder_run(None, None, None, 1, None, None, None) == pdx.PD_ERR_INVALID_ARG
    assert L.predecoder_residual(None, None, None, None, 1, None) == pdx.PD_ERR_INVALID_ARG
    assert L.predecoder_unpack(None, None, None, 1, None) == pdx.PD_ERR_INVALID_ARG
    assert L.predecoder_num_stages(None) == -1
    L.predecoder_destroy(None)


def _create_ex(weights, d, T, layers, layout, first=0, last=0, dtype=pdx.DTYPE_BF16, max_batch=2):
    L = pdx.lib()
    w = np.ascontiguousarray(weights, dtype=np.float32)
    opts = pdx.Options(layout, first, last)
    h = ctypes.c_void_p()
    st = L.predecoder_create_ex(w.ctypes.data_as(ctypes.c_void_p), w.size, d, T, pdx._layers(layers),
                                len(layers), dtype, max_batch, ctypes.byref(opts), ctypes.byref(h))
    if st == pdx.PD_OK:
        L.predecoder_destroy(h)
    return st


PAPER = workload.paper_layer_spec([64, 64, 4], [3, 3, 3])
WP = workload.he_normal_weights(PAPER, 0)


@pytest.mark.parametrize("case", [
    dict(layout=2),                                          # unknown layout
    dict(first=3), dict(last=-1),                            # unknown basis
    dict(layout=pdx.LAYOUT_PLAQUETTE, layers=LAYERS, weights=W, first=pdx.BOUNDARY_Z),  # nothing to clear
    dict(layers=LAYERS, weights=W),                          # paper layout takes 4 input channels
    dict(layout=pdx.LAYOUT_PLAQUETTE),                       # plaquette layout takes 2
])
def test_create_ex_rejects_misuse(case):
    args = dict(weights=WP, d=5, T=3, layers=PAPER, layout=pdx.LAYOUT_PAPER)
    args.update(case)
    assert _create_ex(**args) == pdx.PD_ERR_INVALID_ARG


@pytest.mark.parametrize("layers,dtype", [
    (workload.paper_model_layers(1), pdx.DTYPE_FP32),                  # fp32 on the paper layout
    (workload.paper_layer_spec([256, 256, 4], [3, 3, 1]), pdx.DTYPE_BF16),  # width 256 with a 1x1x1 head
    (workload.paper_layer_spec([192, 4], [3, 3]), pdx.DTYPE_BF16),     # width 192
    (workload.paper_model_layers(3), pdx.DTYPE_FP8),                   # 5x5x5 kernels in fp8
    (workload.paper_layer_spec([128, 128, 4], [5, 3, 3]), pdx.DTYPE_BF16),  # 5x5x5 mixed with 3x3x3
    (workload.paper_layer_spec([128, 128, 4], [5, 5, 1]), pdx.DTYPE_BF16),  # 5x5x5 with a 1x1x1 head
    (workload.paper_layer_spec([256, 4], [5, 5]), pdx.DTYPE_BF16),     # 5x5x5 at width 256
    (workload.paper_layer_spec([64, 4], [5, 5]), pdx.DTYPE_BF16),      # one 5x5x5 hidden layer
    (workload.paper_layer_spec([64, 128, 4], [5, 5, 5]), pdx.DTYPE_BF16),  # 5x5x5 widths that change
])
def test_create_ex_unsupported_models(layers, dtype):
    w = np.zeros(pdx.weight_count(layers), np.float32)
    assert _create_ex(w, 5, 3, layers, pdx.LAYOUT_PAPER, dtype=dtype) == pdx.PD_ERR_UNSUPPORTED


@pytest.mark.skipif(gpu_available(), reason="checks the no-device error path")
def test_create_ex_without_device_reports_device_error():
    assert _create_ex(WP, 5, 3, PAPER, pdx.LAYOUT_PAPER, pdx.BOUNDARY_Z, pdx.BOUNDARY_X) == pdx.PD_ERR_DEVICE


@pytest.mark.skipif(gpu_available(), reason="checks the no-device error path")
def test_model3_passes_validation():
    """Model 3 of Table models (5x5x5 kernels) in bf16 on the paper layout is
    supported: create gets as far as the device check."""
    layers = workload.paper_model_layers(3)
    w = np.zeros(pdx.weight_count(layers), np.float32)
    assert _create_ex(w, 13, 13, layers, pdx.LAYOUT_PAPER, pdx.BOUNDARY_Z, pdx.BOUNDARY_Z) == pdx.PD_ERR_DEVICE


# ---- residual networks (Model 6) ----

def _create_resnet(weights, d, T, blocks, layout=pdx.LAYOUT_PAPER, dtype=pdx.DTYPE_BF16, n_weights=None):
    L = pdx.lib()
    w = np.ascontiguousarray(weights, dtype=np.float32)
    opts = pdx.Options(layout, 0, 0)
    h = ctypes.c_void_p()
    st = L.predecoder_create_resnet(w.ctypes.data_as(ctypes.c_void_p), w.size if n_weights is None else n_weights,
                                    d, T, pdx._blocks(blocks), len(blocks), dtype, 2, ctypes.byref(opts),
                                    ctypes.byref(h))
    if st == pdx.PD_OK:
        L.predecoder_destroy(h)
    return st


def test_resnet_weight_count_matches_oracle():
    import oracle
    for blocks in (workload.MODEL6_BLOCKS, workload.resnet_blocks([64, 64, 64]),
                   [(4, 64, 64, 1), (64, 128, 128, 1), (128, 128, 4, 1)]):
        assert pdx.resnet_weight_count(blocks) == oracle.resnet_weight_count(blocks)
    assert pdx.resnet_weight_count([]) == 0


RB = workload.resnet_blocks([64, 64, 64])
RW = workload.resnet_weights(RB, 0)


@pytest.mark.parametrize("blocks,n_weights", [
    ([(2, 64, 64, 1), (64, 64, 4, 1)], None),          # paper layout takes 4 input channels
    ([(4, 64, 64, 1), (64, 64, 5, 1)], None),          # 4 outputs
    ([(4, 64, 64, 1), (32, 64, 4, 1)], None),          # broken chain
    ([(4, 64, 64, 7), (64, 64, 4, 1)], None),          # unknown activation
    (RB, RW.size - 1),                                 # weight count
])
def test_create_resnet_rejects_misuse(blocks, n_weights):
    w = np.zeros(max(pdx.resnet_weight_count(blocks), 1), np.float32) if n_weights is None else RW
    assert _create_resnet(w, 5, 3, blocks, n_weights=n_weights) == pdx.PD_ERR_INVALID_ARG


@pytest.mark.parametrize("blocks,dtype", [
    (RB, pdx.DTYPE_FP32),                               # bf16 and fp8 only
    # fp8: a projection in a middle block (its projection kernel is bf16 only)
    ([(4, 64, 64, 1), (64, 128, 128, 1), (128, 128, 4, 1)], pdx.DTYPE_FP8),
    # fp8: a last-block projection whose input width differs from c_mid
    ([(4, 64, 64, 1), (64, 128, 4, 1)], pdx.DTYPE_FP8),
    ([(4, 96, 96, 1), (96, 96, 4, 1)], pdx.DTYPE_BF16),  # width 96
    ([(4, 64, 128, 1), (128, 128, 4, 1)], pdx.DTYPE_BF16),  # c_out != c_mid inside the network
])
def test_create_resnet_unsupported(blocks, dtype):
    w = np.zeros(pdx.resnet_weight_count(blocks), np.float32)
    assert _create_resnet(w, 5, 3, blocks, dtype=dtype) == pdx.PD_ERR_UNSUPPORTED


@pytest.mark.skipif(gpu_available(), reason="checks the no-device error path")
@pytest.mark.parametrize("dtype", [pdx.DTYPE_BF16, pdx.DTYPE_FP8])
def test_create_resnet_without_device_reports_device_error(dtype):
    assert _create_resnet(RW, 5, 3, RB, dtype=dtype) == pdx.PD_ERR_DEVICE


def test_graph_create_rejects_null_handle():
    import ctypes as c
    g = c.c_void_p()
    assert pdx.lib().predecoder_graph_create(None, None, 1, None, None, None, c.byref(g)) == pdx.PD_ERR_INVALID_ARG
    assert pdx.lib().predecoder_graph_launch(None, None) == pdx.PD_ERR_INVALID_ARG
    pdx.lib().predecoder_graph_destroy(None)
