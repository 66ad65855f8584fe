"""The Python binding rejects buffers the C ABI would overrun, before any
library call (CPU: the checks run on stand-ins that look like device
tensors, on a binding object with no handle behind it): host tensors, wrong
element sizes, non-contiguous or short buffers, and batch sizes below 1.  A
call whose buffers pass reaches the library with a null handle, which
rejects it without touching the device."""
import numpy as np
import pytest
import torch

import paper_2604_12841_amd as pdx
from paper_2604_12841_amd import workload


class FakeDev:
    """Looks like a contiguous device tensor of n elements of `elem` bytes."""

    def __init__(self, n, elem=8, contiguous=True, rows=None):
        self.n, self.elem, self.contig = n, elem, contiguous
        self.shape = (rows if rows is not None else n,)
        self.is_cuda = True

    def is_contiguous(self):
        return self.contig

    def numel(self):
        return self.n

    def element_size(self):
        return self.elem

    def data_ptr(self):
        return 0


def _bare(d=5, T=5, layers=None, blocks=None, dtype=pdx.DTYPE_BF16, layout=pdx.LAYOUT_PLAQUETTE):
    p = object.__new__(pdx.Predecoder)
    p.d, p.T, p.max_batch = d, T, 64
    p.layers = layers if blocks is None else None
    p.blocks = blocks
    p.dtype, p.layout = dtype, layout
    p.grid = d if layout == pdx.LAYOUT_PAPER else d + 1
    p.det_words = -(-T * (d * d - 1) // 64)
    p.flip_words = -(-T * (3 * d * d - 1) // 64)
    p._h = None
    return p


def _run_args(p, B):
    return FakeDev(B * p.det_words, rows=B), FakeDev(B * p.flip_words), FakeDev(B * p.det_words)


def test_host_tensor_rejected():
    p = _bare(layers=workload.layer_spec(2, 64))
    det, flips, res = _run_args(p, 2)
    with pytest.raises(ValueError, match="device"):
        p.run(torch.zeros((2, p.det_words), dtype=torch.int64), flips, res)


def test_short_outputs_rejected():
    p = _bare(layers=workload.layer_spec(2, 64))
    det, flips, res = _run_args(p, 4)
    with pytest.raises(ValueError, match="flips"):
        p.run(det, FakeDev(4 * p.flip_words - 1), res)
    with pytest.raises(ValueError, match="residual"):
        p.run(det, flips, FakeDev(3 * p.det_words))
    with pytest.raises(ValueError, match="logits"):
        p.run(det, flips, res, logits=FakeDev(4 * 4 * p.T * p.grid ** 2 - 1, elem=4))
    with pytest.raises(ValueError, match="det"):  # an explicit batch larger than det holds
        p.run(det, flips, res, batch=5)
    with pytest.raises(ValueError, match="batch"):
        p.run(det, flips, res, batch=0)


def test_element_size_and_layout_rejected():
    p = _bare(layers=workload.layer_spec(2, 64))
    det, flips, res = _run_args(p, 2)
    with pytest.raises(ValueError, match="8"):
        p.run(det, FakeDev(2 * p.flip_words * 2, elem=4), res)
    with pytest.raises(ValueError, match="contiguous"):
        p.run(det, flips, FakeDev(2 * p.det_words, contiguous=False))
    with pytest.raises(ValueError, match="logits"):
        p.run(det, flips, res, logits=FakeDev(2 * 4 * p.T * p.grid ** 2, elem=2))


def test_unpack_and_activations_sizes():
    p = _bare(layers=workload.layer_spec(2, 64))
    det, _, _ = _run_args(p, 3)
    with pytest.raises(ValueError, match="planes"):
        p.unpack(det, FakeDev(3 * p.T * p.grid ** 2 * 2 - 1, elem=2))
    with pytest.raises(ValueError, match="out"):
        p.activations(det, 0, FakeDev(3 * p.T * p.grid ** 2 * 64 - 1, elem=2))
    with pytest.raises(ValueError, match="range"):  # layer 2 is the head
        p.activations(det, 2, FakeDev(3 * p.T * p.grid ** 2 * 64, elem=2))
    q = _bare(layers=workload.layer_spec(3, 64), dtype=pdx.DTYPE_FP8)
    with pytest.raises(ValueError, match="1"):  # fp8 activations are one byte
        q.activations(det, 0, FakeDev(3 * q.T * q.grid ** 2 * 64, elem=2))


def test_resnet_stop_channels():
    blocks = workload.MODEL6_BLOCKS
    p = _bare(d=5, T=5, blocks=blocks, layout=pdx.LAYOUT_PAPER)
    # block 1: conv1 512, projection 512, conv2 512; blocks 2, 3: 512, 512;
    # block 4: conv1 512, projection 4 (conv2 is the output layer)
    assert [p.stop_channels(k) for k in range(9)] == [512] * 8 + [4]
    with pytest.raises(ValueError):
        p.stop_channels(9)
    det, _, _ = _run_args(p, 1)
    with pytest.raises(ValueError, match="out"):
        p.activations(det, 8, FakeDev(p.T * p.grid ** 2 * 4 - 1, elem=2))


def test_stream_run_sizes():
    s = object.__new__(pdx.Stream)
    s.d, s.n_rounds, s.n_streams = 5, 40, 2
    s.det_words = -(-40 * 24 // 64)
    s.flip_words = -(-40 * 74 // 64)
    s._h = None
    with pytest.raises(ValueError, match="flips"):
        s.run(FakeDev(2 * s.det_words), FakeDev(2 * s.flip_words - 1), FakeDev(2 * s.det_words))


def test_valid_buffers_reach_the_library():
    p = _bare(layers=workload.layer_spec(2, 64))
    det, flips, res = _run_args(p, 2)
    with pytest.raises(pdx.PredecoderError) as e:
        p.run(det, flips, res, stream=0)
    assert e.value.status == 1  # PD_ERR_INVALID_ARG: the null handle
