"""The temporal window driver (Sec. VI, parallel windows in time) on the CPU:
the window plan, argument checks of the C ABI, and, with the oracle, the
locality the driver rests on: the network's outputs on a window's core equal
those of one run over the whole stream exactly when the buffer reaches the
receptive-field half-width h = sum (k - 1) / 2 (Eq. ReceptiveFieldFormula),
and not when it falls short."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2604_12841_amd as pdx
from paper_2604_12841_amd import workload


@pytest.mark.parametrize("n,core,buffer", [(1000, 13, 13), (40, 5, 5), (37, 5, 3), (7, 10, 4), (12, 1, 0),
                                           (30, 30, 9), (100, 21, 30)])
def test_window_plan_tiles_the_stream(n, core, buffer):
    plan = pdx.stream_windows(n, core, buffer)
    assert len(plan) == -(-n // core)
    pos = 0
    for k, (start, length, cs, cl) in enumerate(plan):
        assert cs == pos == k * core and cl == min(core, n - cs) and cl >= 1  # cores tile [0, n)
        pos += cl
        assert start == max(0, cs - buffer) and start + length == min(n, cs + cl + buffer)
    assert pos == n


def test_window_plan_rejects_bad_arguments():
    L = pdx.lib()
    for args in [(0, 5, 5), (10, 0, 5), (10, 5, -1)]:
        assert L.predecoder_stream_windows(*args, None, None, None, None, 0) == -1
    arrs = [(ctypes.c_int32 * 1)() for _ in range(4)]
    assert L.predecoder_stream_windows(10, 5, 5, *arrs, 1) == -1  # two windows, room for one


def _create(weights, d, n, core, buffer, layers, dtype=pdx.DTYPE_BF16, n_streams=1):
    w = np.ascontiguousarray(weights, dtype=np.float32)
    h = ctypes.c_void_p()
    st = pdx.lib().predecoder_stream_create(w.ctypes.data_as(ctypes.c_void_p), w.size, d, n, core, buffer,
                                            pdx._layers(layers), len(layers), dtype, n_streams, None,
                                            ctypes.byref(h))
    if st == pdx.PD_OK:
        pdx.lib().predecoder_stream_destroy(h)
    return st


LAYERS = workload.layer_spec(2, 64)
W = workload.he_normal_weights(LAYERS, 0)


@pytest.mark.parametrize("case", [dict(core=0), dict(buffer=-1), dict(n=0), dict(n_streams=0), dict(d=4)])
def test_stream_create_rejects_misuse(case):
    args = dict(weights=W, d=5, n=40, core=5, buffer=5, layers=LAYERS)
    args.update(case)
    assert _create(**args) == pdx.PD_ERR_INVALID_ARG


def test_stream_create_unsupported_length():
    assert _create(W, 5, 2000, 5, 5, LAYERS) == pdx.PD_ERR_UNSUPPORTED


def test_stream_run_rejects_null():
    assert pdx.lib().predecoder_stream_run(None, None, None, None, None) == pdx.PD_ERR_INVALID_ARG
    pdx.lib().predecoder_stream_destroy(None)


def _windowed_oracle(d, n, core, buffer, planes, layers, weights, layout):
    """Oracle outputs stitched from windows of the plan (each window run on its
    own rounds of the planes)."""
    out = None
    for start, length, cs, cl in pdx.stream_windows(n, core, buffer):
        y = oracle.forward(d, length, np.ascontiguousarray(planes[:, :, start:start + length]), layers, weights,
                           False, layout)
        if out is None:
            out = np.zeros((planes.shape[0], y.shape[1], n) + y.shape[3:])
        out[:, :, cs:cs + cl] = y[:, :, cs - start:cs - start + cl]
    return out


@pytest.mark.parametrize("layout", ["plaquette", "paper"])
def test_cores_equal_the_whole_stream_when_the_buffer_covers_the_receptive_field(layout):
    d, n, core = 5, 23, 4
    if layout == "paper":
        layers = workload.paper_layer_spec([16, 16, 4], [3, 3, 3])  # h = 3
        planes = oracle.unpack_paper(d, n, workload.make_inputs(d, n, 2, 0.05, 0.05, 61)[0])
    else:
        layers = workload.layer_spec(2, 16)                          # h = 2 (1x1x1 head)
        planes = oracle.unpack(d, n, workload.make_inputs(d, n, 2, 0.05, 0.05, 61)[0])
    h = sum((k - 1) // 2 for (_, _, k, _) in layers)
    weights = workload.he_normal_weights(layers, 62)
    whole = oracle.forward(d, n, planes, layers, weights, False, layout)
    exact = _windowed_oracle(d, n, core, h, planes, layers, weights, layout)
    np.testing.assert_array_equal(exact, whole)  # same sums in the same order: bit-identical
    short = _windowed_oracle(d, n, core, h - 1, planes, layers, weights, layout)
    assert np.abs(short - whole).max() > 1e-6  # one round short of the receptive field: cores change
