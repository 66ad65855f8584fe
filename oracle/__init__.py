"""CPU oracle of the pre-decoder hot path (arXiv 2604.12841, Sec. IV.B).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg
of the benchmark are the only callers.  The product path never imports this
package; the two share no code.

The arithmetic lives in ``oracle.c`` (plain C, fp64); this module builds it
with gcc on first use, loads it with ctypes and marshals numpy arrays.
Array layouts are channel-major per sample: planes/logits [B][C][T][H][H],
H = d + 1 on the plaquette grid or H = d in the paper's own layout
(``layout="paper"``: four input channels on the D x D data-qubit grid,
Sec. IV.B.1).
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_NATIVE_PATH = os.path.join(_HERE, "liboracle_native.so")
_lib = None
_native = False
# ISO C (no contraction of a * b + c into one rounding), OpenMP over samples
# and output channels
_FLAGS = ["-O3", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-ffp-contract=off"]


def build(force=False, native=False):
    """Compile oracle.c into liboracle.so (portable), or with native=True into
    liboracle_native.so for the CPU it is built on (-march=native; the same
    IEEE operations in the same order, so the same results, only vector
    instructions of that CPU).  The native build is made on the machine that
    times it."""
    path = _NATIVE_PATH if native else _LIB_PATH
    if force or not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
        tmp = path + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc"] + _FLAGS + (["-march=native"] if native else []) + [_SRC, "-o", tmp, "-lm"])
        os.replace(tmp, path)
    return path


def use_native():
    """Build (on this machine) and use the -march=native library from now on
    (the CPU baseline's timing).  Must come before any other oracle call."""
    global _native
    if _lib is not None and not _native:
        raise RuntimeError("the portable oracle library is already loaded")
    build(force=True, native=True)
    _native = True


def _load():
    global _lib
    if _lib is None:
        path = _NATIVE_PATH if _native else build()
        lib = ctypes.CDLL(path)
        i32, i64, vp = ctypes.c_int, ctypes.c_int64, ctypes.c_void_p
        lib.oracle_site_kind.argtypes = [i32, i32, i32]
        lib.oracle_site_kind.restype = i32
        lib.oracle_plaquette_support.argtypes = [i32, i32, i32, vp]
        lib.oracle_plaquette_support.restype = i32
        lib.oracle_stabilizer_order.argtypes = [i32, vp, vp]
        lib.oracle_stabilizer_order.restype = i32
        lib.oracle_det_words.argtypes = [i32, i32]
        lib.oracle_det_words.restype = i64
        lib.oracle_flip_words.argtypes = [i32, i32]
        lib.oracle_flip_words.restype = i64
        lib.oracle_unpack.argtypes = [i32, i32, i32, vp, vp]
        lib.oracle_unpack.restype = None
        lib.oracle_round_bf16.argtypes = [ctypes.c_float]
        lib.oracle_round_bf16.restype = ctypes.c_float
        lib.oracle_gelu_tanh.argtypes = [ctypes.c_double]
        lib.oracle_gelu_tanh.restype = ctypes.c_double
        lib.oracle_weight_count.argtypes = [i32, vp]
        lib.oracle_weight_count.restype = i64
        lib.oracle_forward.argtypes = [i32, i32, i32, vp, i32, vp, vp, i32, vp]
        lib.oracle_forward.restype = None
        lib.oracle_flips_residual.argtypes = [i32, i32, i32, vp, vp, vp, vp]
        lib.oracle_flips_residual.restype = None
        lib.oracle_residual_from_flips.argtypes = [i32, i32, i32, vp, vp, vp]
        lib.oracle_residual_from_flips.restype = None
        lib.oracle_stabilizer_qubit.argtypes = [i32, i32, i32, vp, vp]
        lib.oracle_stabilizer_qubit.restype = i32
        lib.oracle_unpack_paper.argtypes = [i32, i32, i32, vp, i32, i32, vp]
        lib.oracle_unpack_paper.restype = None
        lib.oracle_forward_grid.argtypes = [i32, i32, i32, vp, i32, vp, vp, i32, vp]
        lib.oracle_forward_grid.restype = None
        lib.oracle_forward_grid_fp8_perturbed.argtypes = [i32, i32, i32, vp, i32, vp, vp, ctypes.c_double,
                                                          ctypes.c_uint64, vp]
        lib.oracle_forward_grid_fp8_perturbed.restype = None
        lib.oracle_flips_residual_paper.argtypes = [i32, i32, i32, vp, vp, vp, vp]
        lib.oracle_flips_residual_paper.restype = None
        lib.oracle_resnet_weight_count.argtypes = [i32, vp, i32]
        lib.oracle_resnet_weight_count.restype = i64
        lib.oracle_forward_resnet.argtypes = [i32, i32, i32, vp, i32, vp, vp, i32, vp]
        lib.oracle_forward_resnet.restype = None
        lib.oracle_forward_resnet_fp8_perturbed.argtypes = [i32, i32, i32, vp, i32, vp, vp, ctypes.c_double,
                                                             ctypes.c_uint64, vp]
        lib.oracle_forward_resnet_fp8_perturbed.restype = None
        lib.oracle_conv_sums.argtypes = [i32, i32, i32, vp, i32, i32, i32, vp, vp, vp, i32]
        lib.oracle_conv_sums.restype = None
        lib.oracle_e4m3_value.argtypes = [i32]
        lib.oracle_e4m3_value.restype = ctypes.c_double
        lib.oracle_e4m3_code.argtypes = [ctypes.c_float]
        lib.oracle_e4m3_code.restype = i32
        lib.oracle_round_e4m3.argtypes = [ctypes.c_float]
        lib.oracle_round_e4m3.restype = ctypes.c_double
        lib.oracle_e4m3_scale_exp.argtypes = [ctypes.c_double]
        lib.oracle_e4m3_scale_exp.restype = i32
        _lib = lib
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def det_words(d, T):
    return int(_load().oracle_det_words(d, T))


def flip_words(d, T):
    return int(_load().oracle_flip_words(d, T))


def site_kind(d):
    """[d+1, d+1] int array: 1 = X stabilizer, 2 = Z stabilizer, 0 = none."""
    lib = _load()
    H = d + 1
    return np.array([[lib.oracle_site_kind(d, i, j) for j in range(H)] for i in range(H)], dtype=np.int32)


def plaquette_support(d, i, j):
    """Data qubits (r, c) acted on by the plaquette at grid site (i, j)."""
    rc = np.zeros(8, dtype=np.int32)
    n = _load().oracle_plaquette_support(d, i, j, _ptr(rc))
    return [(int(rc[2 * e]), int(rc[2 * e + 1])) for e in range(n)]


def stabilizer_order(d):
    """(site_of, index_of): compact stabilizer index <-> flattened grid site."""
    H = d + 1
    site_of = np.zeros(d * d - 1, dtype=np.int32)
    index_of = np.zeros(H * H, dtype=np.int32)
    _load().oracle_stabilizer_order(d, _ptr(site_of), _ptr(index_of))
    return site_of, index_of


def unpack(d, T, det):
    """Packed detectors [B][W_det] uint64 -> planes [B][2][T][d+1][d+1] float64."""
    det = np.ascontiguousarray(det, dtype=np.uint64)
    B = det.shape[0]
    H = d + 1
    out = np.zeros((B, 2, T, H, H), dtype=np.float64)
    _load().oracle_unpack(d, T, B, _ptr(det), _ptr(out))
    return out


def round_bf16(x):
    """Elementwise fp32 -> bf16 (round to nearest even) -> fp32."""
    lib = _load()
    x = np.asarray(x, dtype=np.float32)
    return np.array([lib.oracle_round_bf16(float(v)) for v in x.ravel()], dtype=np.float32).reshape(x.shape)


def e4m3_value(code):
    """Value of an OCP E4M3 code (NaN for 0x7f / 0xff)."""
    return float(_load().oracle_e4m3_value(int(code)))


def e4m3_code(x):
    """Elementwise fp32 -> E4M3 code (nearest, ties to even, saturating at 448)."""
    lib = _load()
    x = np.asarray(x, dtype=np.float32)
    return np.array([lib.oracle_e4m3_code(float(v)) for v in x.ravel()], dtype=np.uint8).reshape(x.shape)


def round_e4m3(x):
    """Elementwise fp32 -> E4M3 -> value."""
    lib = _load()
    x = np.asarray(x, dtype=np.float32)
    return np.array([lib.oracle_round_e4m3(float(v)) for v in x.ravel()], dtype=np.float64).reshape(x.shape)


def e4m3_scale_exp(amax):
    """Scale exponent of a weight row in fp8 mode: smallest e with amax / 2^e <= 448."""
    return int(_load().oracle_e4m3_scale_exp(float(amax)))


def gelu_tanh(x):
    lib = _load()
    x = np.asarray(x, dtype=np.float64)
    return np.array([lib.oracle_gelu_tanh(float(v)) for v in x.ravel()], dtype=np.float64).reshape(x.shape)


def weight_count(layers):
    spec = np.array([list(l) for l in layers], dtype=np.int32).ravel()
    return int(_load().oracle_weight_count(len(layers), _ptr(spec)))


def forward(d, T, planes, layers, weights, bf16, layout="plaquette", fp8=False, fp8_sum_eps=None, fp8_sum_seed=0):
    """Network forward.  planes [B][c_in][T][H][H] float64; layers: list of
    (c_in, c_out, k, act); weights: flat fp32.  Returns logits
    [B][c_out_last][T][H][H] float64 (fp32-valued in bf16 and fp8 mode).
    bf16 / fp8 select the quantisation points of that precision (fp8 wins);
    fp8_sum_eps (fp8 only; None: the plain forward): every sum of products
    moved by a hashed u * eps * sum|products|, u in [-1, 1), the pattern
    chosen by fp8_sum_seed (sizes the fp8 parity bounds)."""
    planes = np.ascontiguousarray(planes, dtype=np.float64)
    weights = np.ascontiguousarray(weights, dtype=np.float32)
    spec = np.ascontiguousarray(np.array([list(l) for l in layers], dtype=np.int32).ravel())
    if weights.size != weight_count(layers):
        raise ValueError("weight count mismatch")
    B = planes.shape[0]
    H = d if layout == "paper" else d + 1
    if planes.shape[1:] != (layers[0][0], T, H, H):
        raise ValueError("planes shape mismatch")
    co = layers[-1][1]
    out = np.zeros((B, co, T, H, H), dtype=np.float64)
    if fp8_sum_eps is not None:
        if not fp8:
            raise ValueError("fp8_sum_eps applies to the fp8 forward")
        _load().oracle_forward_grid_fp8_perturbed(H, T, B, _ptr(planes), len(layers), _ptr(spec), _ptr(weights),
                                                  float(fp8_sum_eps), int(fp8_sum_seed), _ptr(out))
    else:
        prec = 2 if fp8 else (1 if bf16 else 0)
        _load().oracle_forward_grid(H, T, B, _ptr(planes), len(layers), _ptr(spec), _ptr(weights), prec,
                                    _ptr(out))
    return out


BOUNDARY = {None: 0, "none": 0, "Z": 1, "X": 2}


def stabilizer_qubit(d, i, j):
    """(kind, r, c): the data qubit the stabilizer at plaquette (i, j) is drawn
    onto in the paper's layout (kind 1 X, 2 Z; (0, -1, -1) for no stabilizer)."""
    r, c = np.zeros(1, np.int32), np.zeros(1, np.int32)
    kind = _load().oracle_stabilizer_qubit(d, i, j, _ptr(r), _ptr(c))
    return (int(kind), int(r[0]), int(c[0])) if kind else (0, -1, -1)


def unpack_paper(d, T, det, first=None, last=None):
    """Packed detectors -> planes [B][4][T][d][d] of the paper's layout
    (x_type, z_type, x_present, z_present); first / last: basis ("Z", "X" or
    None) of the preparation before round 0 / the measurement after round T-1."""
    det = np.ascontiguousarray(det, dtype=np.uint64)
    B = det.shape[0]
    out = np.zeros((B, 4, T, d, d), dtype=np.float64)
    _load().oracle_unpack_paper(d, T, B, _ptr(det), BOUNDARY[first], BOUNDARY[last], _ptr(out))
    return out


def flips_residual_paper(d, T, logits, det):
    """logits [B][4][T][d][d] of the paper's layout + packed det -> (packed flips, packed residual)."""
    logits = np.ascontiguousarray(logits, dtype=np.float64)
    det = np.ascontiguousarray(det, dtype=np.uint64)
    B = logits.shape[0]
    flips = np.zeros((B, flip_words(d, T)), dtype=np.uint64)
    res = np.zeros((B, det_words(d, T)), dtype=np.uint64)
    _load().oracle_flips_residual_paper(d, T, B, _ptr(logits), _ptr(det), _ptr(flips), _ptr(res))
    return flips, res


def flips_residual(d, T, logits, det):
    """logits [B][4][T][H][H] + packed det -> (packed flips, packed residual)."""
    logits = np.ascontiguousarray(logits, dtype=np.float64)
    det = np.ascontiguousarray(det, dtype=np.uint64)
    B = logits.shape[0]
    flips = np.zeros((B, flip_words(d, T)), dtype=np.uint64)
    res = np.zeros((B, det_words(d, T)), dtype=np.uint64)
    _load().oracle_flips_residual(d, T, B, _ptr(logits), _ptr(det), _ptr(flips), _ptr(res))
    return flips, res


def residual_from_flips(d, T, det, flips):
    det = np.ascontiguousarray(det, dtype=np.uint64)
    flips = np.ascontiguousarray(flips, dtype=np.uint64)
    B = det.shape[0]
    res = np.zeros((B, det_words(d, T)), dtype=np.uint64)
    _load().oracle_residual_from_flips(d, T, B, _ptr(det), _ptr(flips), _ptr(res))
    return res


def num_threads():
    """Threads the oracle's parallel loops use."""
    lib = _load()
    lib.oracle_num_threads.restype = ctypes.c_int
    return int(lib.oracle_num_threads())


def set_num_threads(n):
    """Threads for the oracle's parallel loops from now on."""
    lib = _load()
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_num_threads.restype = None
    lib.oracle_set_num_threads(int(n))


def run(d, T, det, layers, weights, bf16, layout="plaquette", first=None, last=None, fp8=False):
    """The whole path: (logits, flips, residual)."""
    if layout == "paper":
        logits = forward(d, T, unpack_paper(d, T, det, first, last), layers, weights, bf16, layout, fp8)
        flips, res = flips_residual_paper(d, T, logits, det)
    else:
        logits = forward(d, T, unpack(d, T, det), layers, weights, bf16, fp8=fp8)
        flips, res = flips_residual(d, T, logits, det)
    return logits, flips, res


def resnet_weight_count(blocks, bn_per_channel=4):
    """Floats of a residual network's weights; blocks: (c_in, c_mid, c_out, act).  bn_per_channel = 4
    (scale, shift, running mean, running variance) as the weights are passed, 2 for the trainable count."""
    spec = np.ascontiguousarray(np.array([list(b) for b in blocks], dtype=np.int32).ravel())
    return int(_load().oracle_resnet_weight_count(len(blocks), _ptr(spec), bn_per_channel))


def forward_resnet(d, T, planes, blocks, weights, bf16, layout="plaquette", acc32=False, fp8=False,
                   fp8_sum_eps=None, fp8_sum_seed=0):
    """Residual network forward (Model 6, Sec. VI, Fig. Model8Representation).  planes [B][c_in][T][H][H];
    blocks: (c_in, c_mid, c_out, act); returns logits [B][4][T][H][H].  acc32 (bf16 only): the conv sums
    in fp32 (sizes the parity tolerance).  fp8: the E4M3 precision points (folded weights per output
    channel, every stored tensor); fp8_sum_eps (test infrastructure) moves every sum by up to that
    fraction of its sum of magnitudes, hashed per fp8_sum_seed (sizes the fp8 parity tolerance)."""
    planes = np.ascontiguousarray(planes, dtype=np.float64)
    weights = np.ascontiguousarray(weights, dtype=np.float32)
    spec = np.ascontiguousarray(np.array([list(b) for b in blocks], dtype=np.int32).ravel())
    if weights.size != resnet_weight_count(blocks):
        raise ValueError("weight count mismatch")
    B = planes.shape[0]
    H = d if layout == "paper" else d + 1
    if planes.shape[1:] != (blocks[0][0], T, H, H) or blocks[-1][2] != 4:
        raise ValueError("planes / blocks mismatch")
    out = np.zeros((B, 4, T, H, H), dtype=np.float64)
    if fp8_sum_eps is not None:
        if not fp8:
            raise ValueError("fp8_sum_eps needs fp8")
        _load().oracle_forward_resnet_fp8_perturbed(H, T, B, _ptr(planes), len(blocks), _ptr(spec), _ptr(weights),
                                                    float(fp8_sum_eps), int(fp8_sum_seed), _ptr(out))
        return out
    prec = 3 if fp8 else ((2 if acc32 else 1) if bf16 else 0)
    _load().oracle_forward_resnet(H, T, B, _ptr(planes), len(blocks), _ptr(spec), _ptr(weights), prec, _ptr(out))
    return out


def conv_sums(x, w, bias, acc32=False):
    """One conv3d of the residual-network forward (cross-correlation, zero
    padding (k-1)/2): x [B][c_in][T][H][H], w [c_out][c_in][k][k][k], bias
    [c_out], all float64 -> [B][c_out][T][H][H]; sums over (c_in, kt, ki, kj)
    in that order, in fp64, or with acc32 each product rounded to fp32 and
    added to an fp32 sum."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    w = np.ascontiguousarray(w, dtype=np.float64)
    bias = np.ascontiguousarray(bias, dtype=np.float64)
    B, ci, T, H, _ = x.shape
    co, k = w.shape[0], w.shape[2]
    if w.shape != (co, ci, k, k, k) or bias.shape != (co,) or k % 2 != 1:
        raise ValueError("conv_sums shapes")
    y = np.zeros((B, co, T, H, H), dtype=np.float64)
    _load().oracle_conv_sums(H, T, B, _ptr(x), ci, co, k, _ptr(w), _ptr(bias), _ptr(y), int(bool(acc32)))
    return y


def run_resnet(d, T, det, blocks, weights, bf16, layout="paper", first=None, last=None, fp8=False):
    """The whole path with a residual network: (logits, flips, residual)."""
    if layout == "paper":
        logits = forward_resnet(d, T, unpack_paper(d, T, det, first, last), blocks, weights, bf16, layout, fp8=fp8)
        flips, res = flips_residual_paper(d, T, logits, det)
    else:
        logits = forward_resnet(d, T, unpack(d, T, det), blocks, weights, bf16, fp8=fp8)
        flips, res = flips_residual(d, T, logits, det)
    return logits, flips, res
