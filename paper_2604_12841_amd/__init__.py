"""MI355X (gfx950) pre-decoder for the rotated surface code (arXiv 2604.12841).

Thin ctypes binding over the C ABI in include/predecoder.h: it only marshals
arguments.  Every step of the path (unpack, conv layers, head, threshold,
residual, bit repack) runs in the HIP kernels of libpredecoder.so, which is
built in-tree by ``paper_2604_12841_amd.build``.  There is no CPU fallback:
if the library is missing, loading it raises.

Device buffers are torch tensors on the GPU (torch is used only for device
memory and streams); streams are passed as their raw hipStream_t handles.
"""
import ctypes
import os

__all__ = ["Predecoder", "Stream", "stream_windows", "PredecoderError", "Options", "lib", "det_words", "flip_words", "weight_count",
           "status_string", "ACT_NONE", "ACT_GELU_TANH", "ACT_RELU", "DTYPE_FP32", "DTYPE_BF16", "DTYPE_FP8",
           "LAYOUT_PLAQUETTE", "LAYOUT_PAPER", "BOUNDARY_NONE", "BOUNDARY_Z", "BOUNDARY_X", "LIB_PATH",
           "EXPORTS"]

ACT_NONE, ACT_GELU_TANH, ACT_RELU = 0, 1, 2
DTYPE_FP32, DTYPE_BF16, DTYPE_FP8 = 0, 1, 2
_DTYPES = {"fp32": DTYPE_FP32, "bf16": DTYPE_BF16, "fp8": DTYPE_FP8}
LAYOUT_PLAQUETTE, LAYOUT_PAPER = 0, 1
BOUNDARY_NONE, BOUNDARY_Z, BOUNDARY_X = 0, 1, 2
_LAYOUTS = {"plaquette": LAYOUT_PLAQUETTE, "paper": LAYOUT_PAPER}
_BOUNDARIES = {None: BOUNDARY_NONE, "none": BOUNDARY_NONE, "Z": BOUNDARY_Z, "X": BOUNDARY_X}
PD_OK, PD_ERR_INVALID_ARG, PD_ERR_UNSUPPORTED, PD_ERR_OUT_OF_MEMORY, PD_ERR_DEVICE, PD_ERR_TOO_LARGE = range(6)
STATIC_SCRATCH_BYTES = 64 << 20  # PD_STATIC_SCRATCH_BYTES

# PD_LIBRARY: another build of the library to load (the host-sanitizer build
# of build.py --sanitize); by default the in-tree libpredecoder.so
LIB_PATH = os.environ.get("PD_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                         "libpredecoder.so")

# Every symbol declared in include/predecoder.h.
EXPORTS = ("predecoder_create", "predecoder_create_ex", "predecoder_run", "predecoder_residual", "predecoder_unpack",
           "predecoder_activations",
           "predecoder_num_stages", "predecoder_stage_times", "predecoder_destroy",
           "predecoder_status_string", "predecoder_det_words", "predecoder_flip_words",
           "predecoder_weight_count", "predecoder_stream_windows", "predecoder_stream_create",
           "predecoder_stream_run", "predecoder_stream_destroy", "predecoder_resnet_weight_count",
           "predecoder_create_resnet", "predecoder_graph_create", "predecoder_graph_launch",
           "predecoder_graph_destroy", "predecoder_run_static", "predecoder_peak_mfma", "predecoder_peak_copy")


class PredecoderError(RuntimeError):
    def __init__(self, status, what):
        super().__init__("%s: %s (status %d)" % (what, status_string(status), status))
        self.status = status


class Layer(ctypes.Structure):
    _fields_ = [("c_in", ctypes.c_int32), ("c_out", ctypes.c_int32), ("k", ctypes.c_int32),
                ("act", ctypes.c_int32)]


class Block(ctypes.Structure):
    _fields_ = [("c_in", ctypes.c_int32), ("c_mid", ctypes.c_int32), ("c_out", ctypes.c_int32),
                ("act", ctypes.c_int32)]


class Options(ctypes.Structure):
    _fields_ = [("layout", ctypes.c_int32), ("first_round", ctypes.c_int32), ("last_round", ctypes.c_int32)]


_lib = None


def lib():
    """The loaded libpredecoder.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libpredecoder.so is not built: run paper_2604_12841_amd/build.py")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        LP = ctypes.POINTER(Layer)
        L.predecoder_create.argtypes = [vp, sz, i32, i32, LP, i32, i32, i32, ctypes.POINTER(vp)]
        L.predecoder_create.restype = i32
        L.predecoder_create_ex.argtypes = [vp, sz, i32, i32, LP, i32, i32, i32, ctypes.POINTER(Options),
                                           ctypes.POINTER(vp)]
        L.predecoder_create_ex.restype = i32
        L.predecoder_run.argtypes = [vp, vp, vp, i32, vp, vp, vp]
        L.predecoder_run.restype = i32
        L.predecoder_residual.argtypes = [vp, vp, vp, vp, i32, vp]
        L.predecoder_residual.restype = i32
        L.predecoder_unpack.argtypes = [vp, vp, vp, i32, vp]
        L.predecoder_unpack.restype = i32
        L.predecoder_activations.argtypes = [vp, vp, vp, i32, i32, vp]
        L.predecoder_activations.restype = i32
        L.predecoder_num_stages.argtypes = [vp]
        L.predecoder_num_stages.restype = i32
        L.predecoder_stage_times.argtypes = [vp, vp, vp, i32, vp, vp, i32, ctypes.POINTER(ctypes.c_float)]
        L.predecoder_stage_times.restype = i32
        L.predecoder_destroy.argtypes = [vp]
        L.predecoder_destroy.restype = None
        L.predecoder_status_string.argtypes = [i32]
        L.predecoder_status_string.restype = ctypes.c_char_p
        L.predecoder_det_words.argtypes = [i32, i32]
        L.predecoder_det_words.restype = i64
        L.predecoder_flip_words.argtypes = [i32, i32]
        L.predecoder_flip_words.restype = i64
        L.predecoder_weight_count.argtypes = [LP, i32]
        L.predecoder_weight_count.restype = sz
        IP = ctypes.POINTER(i32)
        L.predecoder_stream_windows.argtypes = [i32, i32, i32, IP, IP, IP, IP, i32]
        L.predecoder_stream_windows.restype = i32
        L.predecoder_stream_create.argtypes = [vp, sz, i32, i32, i32, i32, LP, i32, i32, i32, ctypes.POINTER(Options),
                                               ctypes.POINTER(vp)]
        L.predecoder_stream_create.restype = i32
        L.predecoder_stream_run.argtypes = [vp, vp, vp, vp, vp]
        L.predecoder_stream_run.restype = i32
        L.predecoder_stream_destroy.argtypes = [vp]
        L.predecoder_stream_destroy.restype = None
        BP = ctypes.POINTER(Block)
        L.predecoder_resnet_weight_count.argtypes = [BP, i32]
        L.predecoder_resnet_weight_count.restype = sz
        L.predecoder_create_resnet.argtypes = [vp, sz, i32, i32, BP, i32, i32, i32, ctypes.POINTER(Options),
                                               ctypes.POINTER(vp)]
        L.predecoder_create_resnet.restype = i32
        L.predecoder_graph_create.argtypes = [vp, vp, i32, vp, vp, vp, ctypes.POINTER(vp)]
        L.predecoder_graph_create.restype = i32
        L.predecoder_graph_launch.argtypes = [vp, vp]
        L.predecoder_graph_launch.restype = i32
        L.predecoder_graph_destroy.argtypes = [vp]
        L.predecoder_graph_destroy.restype = None
        L.predecoder_run_static.argtypes = [vp, vp, vp, i32, vp, vp, vp]
        L.predecoder_run_static.restype = i32
        L.predecoder_peak_mfma.argtypes = [vp, i32, vp, i32, i32, vp]
        L.predecoder_peak_mfma.restype = i32
        L.predecoder_peak_copy.argtypes = [vp, vp, vp, sz]
        L.predecoder_peak_copy.restype = i32
        _lib = L
    return _lib


def status_string(status):
    return lib().predecoder_status_string(int(status)).decode()


def det_words(d, T):
    return int(lib().predecoder_det_words(d, T))


def flip_words(d, T):
    return int(lib().predecoder_flip_words(d, T))


def _layers(layers):
    arr = (Layer * len(layers))()
    for i, l in enumerate(layers):
        arr[i] = Layer(*[int(v) for v in l])
    return arr


def _blocks(blocks):
    arr = (Block * len(blocks))()
    for i, b in enumerate(blocks):
        arr[i] = Block(*[int(v) for v in b])
    return arr


def resnet_weight_count(blocks):
    return int(lib().predecoder_resnet_weight_count(_blocks(blocks), len(blocks)))


def weight_count(layers):
    return int(lib().predecoder_weight_count(_layers(layers), len(layers)))


def _ptr(t, what="buffer", nbytes=0, elem=None):
    """Raw device pointer of a tensor (or None), after checking that it is a
    contiguous device tensor with elements of `elem` bytes (one of them, if a
    tuple) and at least `nbytes` bytes: the kernels behind the C ABI read and
    write that many bytes and cannot check a raw pointer themselves."""
    if t is None:
        return None
    if not getattr(t, "is_cuda", False):
        raise ValueError("%s must be a device (GPU) tensor" % what)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % what)
    if elem is not None and t.element_size() not in (elem if isinstance(elem, tuple) else (elem,)):
        raise ValueError("%s has %d-byte elements, expected %s" % (what, t.element_size(), elem))
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError("%s holds %d bytes, the call uses %d" % (what, have, nbytes))
    return ctypes.c_void_p(t.data_ptr())


def _batch(batch, first):
    """The batch of a call: given, or the leading dimension of `first`."""
    b = int(first.shape[0]) if batch is None else int(batch)
    if b < 1:
        raise ValueError("batch must be >= 1")
    return b


def _stream(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


class Predecoder:
    """One pre-decoder handle: weights, workspace and tables for (d, T, max_batch)."""

    def __init__(self, weights, d, T, layers, dtype="bf16", max_batch=1, layout="plaquette", first=None,
                 last=None, blocks=None):
        """layout: "plaquette" or "paper" (Sec. IV.B.1); first / last: basis ("Z", "X" or None) of the
        preparation before round 0 / the measurement after round T-1 (paper layout).  blocks (with
        layers None): a residual network of (c_in, c_mid, c_out, act) blocks (Model 6)."""
        import numpy as np
        w = np.ascontiguousarray(np.asarray(weights, dtype=np.float32))
        self.d, self.T, self.max_batch = d, T, max_batch
        self.layers = [tuple(l) for l in layers] if layers is not None else None
        self.blocks = [tuple(b) for b in blocks] if blocks is not None else None
        self.dtype = _DTYPES[dtype] if isinstance(dtype, str) else int(dtype)
        self.layout = _LAYOUTS[layout] if isinstance(layout, str) else int(layout)
        self.grid = d if self.layout == LAYOUT_PAPER else d + 1
        self.det_words = det_words(d, T)
        self.flip_words = flip_words(d, T)
        opts = Options(self.layout, _BOUNDARIES[first] if not isinstance(first, int) else first,
                       _BOUNDARIES[last] if not isinstance(last, int) else last)
        h = ctypes.c_void_p()
        if blocks is not None:
            st = lib().predecoder_create_resnet(w.ctypes.data_as(ctypes.c_void_p), w.size, d, T, _blocks(blocks),
                                                len(blocks), self.dtype, max_batch, ctypes.byref(opts),
                                                ctypes.byref(h))
        else:
            st = lib().predecoder_create_ex(w.ctypes.data_as(ctypes.c_void_p), w.size, d, T, _layers(layers),
                                            len(layers), self.dtype, max_batch, ctypes.byref(opts), ctypes.byref(h))
        if st != PD_OK:
            raise PredecoderError(st, "predecoder_create")
        self._h = h

    def _check(self, st, what):
        if st != PD_OK:
            raise PredecoderError(st, what)

    # ---- argument marshalling: every buffer checked against what the call
    # reads or writes for `batch` samples ----

    def _io(self, det, flips, residual, logits, batch):
        """Pointers of a run's buffers (det, flips, residual, logits or None)."""
        return (_ptr(det, "det", batch * self.det_words * 8, 8),
                _ptr(flips, "flips", batch * self.flip_words * 8, 8),
                _ptr(residual, "residual", batch * self.det_words * 8, 8),
                _ptr(logits, "logits", batch * 4 * self.T * self.grid ** 2 * 4, 4))

    def stop_channels(self, layer):
        """Channels of what predecoder_activations returns for `layer`: a
        hidden layer's width, or for a residual network the width of conv
        number `layer` (per block: conv1, the projection if any, conv2)."""
        if self.blocks is None:
            if not 0 <= layer < len(self.layers) - 1:
                raise ValueError("layer out of range")
            return self.layers[layer][1]
        outs = []
        for ci, cm, co, _a in self.blocks:
            outs += [cm] + ([co] if ci != co else []) + [co]
        if not 0 <= layer < len(outs) - 1:
            raise ValueError("layer out of range")
        return outs[layer]

    def run(self, det, flips, residual, logits=None, batch=None, stream=None):
        """det [B][W_det] uint64-valued int64 tensor -> flips [B][W_flip], residual [B][W_det] (in place)."""
        batch = _batch(batch, det)
        pd, pf, pr, pl = self._io(det, flips, residual, logits, batch)
        self._check(lib().predecoder_run(self._h, _stream(stream), pd, batch, pf, pr, pl), "predecoder_run")

    def run_static(self, det, flips, residual, logits=None, batch=None, stream=None):
        """run() with the workspace in the library's static device array (allocates nothing; calls that
        overlap on one device race)."""
        batch = _batch(batch, det)
        pd, pf, pr, pl = self._io(det, flips, residual, logits, batch)
        self._check(lib().predecoder_run_static(self._h, _stream(stream), pd, batch, pf, pr, pl),
                    "predecoder_run_static")

    def residual(self, det, flips, residual, batch=None, stream=None):
        batch = _batch(batch, det)
        pd, pf, pr, _ = self._io(det, flips, residual, None, batch)
        self._check(lib().predecoder_residual(self._h, _stream(stream), pd, pf, batch, pr), "predecoder_residual")

    def unpack(self, det, planes, batch=None, stream=None):
        """det -> planes [B][T][H][H][c_in] (bf16 bits, or fp32 on an fp32 handle)."""
        batch = _batch(batch, det)
        c_in = 4 if self.layout == LAYOUT_PAPER else 2
        elem = 4 if self.dtype == DTYPE_FP32 else 2
        pd = _ptr(det, "det", batch * self.det_words * 8, 8)
        pp = _ptr(planes, "planes", batch * self.T * self.grid ** 2 * c_in * elem, elem)
        self._check(lib().predecoder_unpack(self._h, _stream(stream), pd, batch, pp), "predecoder_unpack")

    def activations(self, det, layer, out, batch=None, stream=None):
        """Output activations of hidden layer `layer` (residual networks: of conv number `layer`) -> out
        [B][T][H][H][c_out] (bf16 bits as int16, E4M3 codes as uint8)."""
        batch = _batch(batch, det)
        elem = 1 if self.dtype == DTYPE_FP8 else 2
        pd = _ptr(det, "det", batch * self.det_words * 8, 8)
        po = _ptr(out, "out", batch * self.T * self.grid ** 2 * self.stop_channels(layer) * elem, elem)
        self._check(lib().predecoder_activations(self._h, _stream(stream), pd, batch, layer, po),
                    "predecoder_activations")

    def graph(self, det, flips, residual, logits=None, batch=None):
        """Records one run with these buffers; returns a Graph to replay it."""
        batch = _batch(batch, det)
        pd, pf, pr, pl = self._io(det, flips, residual, logits, batch)
        g = ctypes.c_void_p()
        self._check(lib().predecoder_graph_create(self._h, pd, batch, pf, pr, pl, ctypes.byref(g)),
                    "predecoder_graph_create")
        return Graph(g)

    @property
    def num_stages(self):
        return int(lib().predecoder_num_stages(self._h))

    def stage_times(self, det, flips, residual, n_iter, batch=None, stream=None):
        """Mean milliseconds of each stage over n_iter runs (blocks until done)."""
        batch = _batch(batch, det)
        pd, pf, pr, _ = self._io(det, flips, residual, None, batch)
        out = (ctypes.c_float * self.num_stages)()
        self._check(lib().predecoder_stage_times(self._h, _stream(stream), pd, batch, pf, pr, n_iter, out),
                    "predecoder_stage_times")
        return list(out)

    def close(self):
        if getattr(self, "_h", None):
            lib().predecoder_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def peak_mfma(dtype, operands, iters, n_workgroups, out, stream=None):
    """Back-to-back matrix instructions (predecoder_peak_mfma): operands, 4096-byte device tensor; out,
    n_workgroups x 256 float32 device tensor.  Returns the FLOPs launched."""
    dt = _DTYPES[dtype] if isinstance(dtype, str) else int(dtype)
    po = _ptr(operands, "operands", 4096)
    pout = _ptr(out, "out", n_workgroups * 256 * 4, 4)
    st = lib().predecoder_peak_mfma(_stream(stream), dt, po, int(iters), int(n_workgroups), pout)
    if st != PD_OK:
        raise PredecoderError(st, "predecoder_peak_mfma")
    return n_workgroups * 4 * iters * 4 * (131072 if dt == DTYPE_FP8 else 32768)


def peak_copy(src, dst, nbytes, stream=None):
    """dst[:nbytes] = src[:nbytes] with the library's copy kernel (predecoder_peak_copy)."""
    ps, pd = _ptr(src, "src", nbytes), _ptr(dst, "dst", nbytes)
    st = lib().predecoder_peak_copy(_stream(stream), ps, pd, int(nbytes))
    if st != PD_OK:
        raise PredecoderError(st, "predecoder_peak_copy")


def stream_windows(n_rounds, core, buffer):
    """The temporal window plan: list of (start, length, core_start, core_length)."""
    L = lib()
    n = L.predecoder_stream_windows(n_rounds, core, buffer, None, None, None, None, 0)
    if n < 0:
        raise ValueError("invalid window plan")
    arrs = [(ctypes.c_int32 * n)() for _ in range(4)]
    L.predecoder_stream_windows(n_rounds, core, buffer, *arrs, n)
    return [tuple(int(a[k]) for a in arrs) for k in range(n)]


class Stream:
    """Temporal window driver over n_streams streams of n_rounds rounds (Sec. VI, parallel windows in time)."""

    def __init__(self, weights, d, n_rounds, layers, core, buffer, dtype="bf16", n_streams=1, layout="plaquette",
                 first=None, last=None):
        import numpy as np
        w = np.ascontiguousarray(np.asarray(weights, dtype=np.float32))
        self.d, self.n_rounds, self.n_streams = d, n_rounds, n_streams
        self.det_words = det_words(d, n_rounds)
        self.flip_words = flip_words(d, n_rounds)
        lay = _LAYOUTS[layout] if isinstance(layout, str) else int(layout)
        opts = Options(lay, _BOUNDARIES[first] if not isinstance(first, int) else first,
                       _BOUNDARIES[last] if not isinstance(last, int) else last)
        dt = _DTYPES[dtype] if isinstance(dtype, str) else int(dtype)
        h = ctypes.c_void_p()
        st = lib().predecoder_stream_create(w.ctypes.data_as(ctypes.c_void_p), w.size, d, n_rounds, core, buffer,
                                            _layers(layers), len(layers), dt, n_streams, ctypes.byref(opts),
                                            ctypes.byref(h))
        if st != PD_OK:
            raise PredecoderError(st, "predecoder_stream_create")
        self._h = h

    def run(self, det, flips, residual, stream=None):
        """det [n_streams][W_det] -> flips [n_streams][W_flip], residual [n_streams][W_det] (device, in place)."""
        n = self.n_streams
        pd = _ptr(det, "det", n * self.det_words * 8, 8)
        pf = _ptr(flips, "flips", n * self.flip_words * 8, 8)
        pr = _ptr(residual, "residual", n * self.det_words * 8, 8)
        st = lib().predecoder_stream_run(self._h, _stream(stream), pd, pf, pr)
        if st != PD_OK:
            raise PredecoderError(st, "predecoder_stream_run")

    def close(self):
        if getattr(self, "_h", None):
            lib().predecoder_stream_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Graph:
    """A recorded predecoder_run (Predecoder.graph)."""

    def __init__(self, handle):
        self._h = handle

    def launch(self, stream=None):
        st = lib().predecoder_graph_launch(self._h, _stream(stream))
        if st != PD_OK:
            raise PredecoderError(st, "predecoder_graph_launch")

    def close(self):
        if getattr(self, "_h", None):
            lib().predecoder_graph_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
