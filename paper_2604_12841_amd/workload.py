"""Seeded synthetic workloads for the pre-decoder (inputs only, no method arithmetic).

Holds the five configurations the path is measured on, He-normal weight draws,
the phenomenological noise model (independent X and Z data-qubit flips with
probability p per round, independent measurement flips with probability q per
stabilizer and round), the detector events that noise produces, and the
LSB-first bit packing of the C ABI.  Both the GPU path's tests/benchmark and
the CPU oracle consume these arrays; neither side shares code with the other.

The stabilizer layout used to turn sampled errors into detector events is
built here from data-qubit coordinates (an ancilla at half-integer position
(r - 1/2, c - 1/2) checks the data qubits at (r - 1/2 +- 1/2, c - 1/2 +- 1/2)),
independently of both the oracle and the GPU tables; it matches the rotated
code of Sec. III (X_L horizontal, Z_L vertical) and the compact detector order
of the ABI (X ancillas row-major, then Z ancillas row-major).

Detector events follow Sec. IV.B.1: d_{i,k} = s_{i,k} XOR s_{i,k-1} with
s_{i,-1} = 0, where the reported outcome s_{i,k} is the parity of the
accumulated data errors on the stabilizer's support XOR that round's
measurement error.
"""
import numpy as np

GELU_TANH = 1
RELU = 2
NONE = 0

# Workload table: distance, rounds, batch, hidden conv3d layers x width,
# precision, phenomenological error rates.  Weight seed 1000+id, noise seed 2000+id.
CONFIGS = {
    1: dict(d=5, T=5, batch=64, n_hidden=4, width=32, dtype="fp32", p=0.003, q=0.003),
    2: dict(d=9, T=9, batch=1024, n_hidden=6, width=64, dtype="bf16", p=0.005, q=0.005),
    3: dict(d=13, T=13, batch=4096, n_hidden=8, width=128, dtype="bf16", p=0.003, q=0.003),
    4: dict(d=25, T=25, batch=1, n_hidden=6, width=64, dtype="bf16", p=0.002, q=0.002),
    5: dict(d=31, T=31, batch=256, n_hidden=8, width=128, dtype="bf16", p=0.004, q=0.004),
}

BIAS_STD = 0.35


def layer_spec(n_hidden, width, act=GELU_TANH, c_in=2, c_out=4):
    """n_hidden 3x3x3 conv layers (c_in -> width -> ... -> width) then a 1x1x1 head to c_out."""
    layers = []
    ci = c_in
    for _ in range(n_hidden):
        layers.append((ci, width, 3, act))
        ci = width
    layers.append((ci, c_out, 1, NONE))
    return layers


# The models of Table models (Sec. VI) in the paper's own layout: four input
# channels (x_type, z_type, x_present, z_present on the D x D grid), the
# listed filters and kernel sizes per conv layer, the last layer (4 filters)
# without activation.
PAPER_MODELS = {
    1: ([128, 128, 128, 4], [3, 3, 3, 3]),
    2: ([256, 256, 256, 4], [3, 3, 3, 3]),
    3: ([128, 128, 128, 4], [5, 5, 5, 5]),
    4: ([128, 128, 128, 128, 128, 4], [3, 3, 3, 3, 3, 3]),
    5: ([256, 256, 256, 256, 256, 4], [3, 3, 3, 3, 3, 3]),
}


def paper_model_layers(model, act=GELU_TANH):
    filters, kernels = PAPER_MODELS[model]
    return paper_layer_spec(filters, kernels, act)


def paper_layer_spec(filters, kernels, act=GELU_TANH, c_in=4):
    layers = []
    ci = c_in
    for n, (co, k) in enumerate(zip(filters, kernels)):
        layers.append((ci, co, k, NONE if n == len(filters) - 1 else act))
        ci = co
    return layers


# Model 6 (Sec. VI, Fig. Model8Representation): four residual blocks
# (c_in, c_mid, c_out, act), two 3x3x3 convs with BatchNorm each; the first
# expands 4 -> 512 and the last compresses 512 -> 4, both with a 1x1x1
# projection shortcut.
MODEL6_BLOCKS = [(4, 512, 512, GELU_TANH), (512, 512, 512, GELU_TANH), (512, 512, 512, GELU_TANH),
                 (512, 512, 4, GELU_TANH)]


def resnet_blocks(widths, c_in=4, act=GELU_TANH):
    """Blocks of a residual network with hidden width `widths[k]` in block k
    and 4 output channels: (c_in, c_mid, c_out, act)."""
    blocks, ci = [], c_in
    for k, w in enumerate(widths):
        co = 4 if k == len(widths) - 1 else w
        blocks.append((ci, w, co, act))
        ci = co
    return blocks


def resnet_weights(blocks, seed, bias_std=BIAS_STD):
    """Random weights of a residual network in the order the C ABI takes
    them, per block: conv1 w, b; BatchNorm1 scale, shift, running mean,
    running variance; conv2 w, b; BatchNorm2 (same four); projection w, b
    when c_in != c_out.  Convs He-normal, biases N(0, bias_std^2), BatchNorm
    scale N(1, 0.1^2), shift N(0, 0.1^2), mean N(0, 0.1^2), variance
    U(0.5, 1.5)."""
    rng = np.random.default_rng(seed)
    parts = []
    for ci, cm, co, _act in blocks:
        for cin, cout in ((ci, cm), (cm, co)):
            parts.append(rng.standard_normal(cout * cin * 27) * np.sqrt(2.0 / (cin * 27)))
            parts.append(rng.standard_normal(cout) * bias_std)
            parts.append(1.0 + 0.1 * rng.standard_normal(cout))
            parts.append(0.1 * rng.standard_normal(cout))
            parts.append(0.1 * rng.standard_normal(cout))
            parts.append(rng.uniform(0.5, 1.5, cout))
        if ci != co:
            parts.append(rng.standard_normal(co * ci) * np.sqrt(2.0 / ci))
            parts.append(rng.standard_normal(co) * bias_std)
    return np.concatenate(parts).astype(np.float32)


def config_layers(cfg_id, act=GELU_TANH):
    c = CONFIGS[cfg_id]
    return layer_spec(c["n_hidden"], c["width"], act)


def he_normal_weights(layers, seed, bias_std=BIAS_STD):
    """Per layer: W ~ N(0, 2 / (c_in k^3)) of shape [c_out][c_in][k][k][k], then
    b ~ N(0, bias_std^2) of shape [c_out]; concatenated, fp32."""
    rng = np.random.default_rng(seed)
    parts = []
    for (ci, co, k, _act) in layers:
        w = rng.standard_normal((co, ci, k, k, k)) * np.sqrt(2.0 / (ci * k ** 3))
        b = rng.standard_normal(co) * bias_std
        parts.append(w.astype(np.float32).ravel())
        parts.append(b.astype(np.float32))
    return np.concatenate(parts)


def config_weights(cfg_id, act=GELU_TANH):
    return he_normal_weights(config_layers(cfg_id, act), 1000 + cfg_id)


# ---------------------------------------------------------------------------
# Code layout from data-qubit coordinates
# ---------------------------------------------------------------------------

def ancillas(d):
    """Ancillas of the distance-d rotated surface code as (kind, r, c, support),
    kind 'X' or 'Z', at half-integer position (r - 1/2, c - 1/2) for
    0 <= r, c <= d, support = list of data-qubit indices q = row * d + col.
    Checkerboard colouring with X where r + c is even; a bulk ancilla has four
    neighbours; on the boundary only X ancillas on the left/right edges and Z
    ancillas on the top/bottom edges are kept, each with two neighbours."""
    out = []
    for r in range(d + 1):
        for c in range(d + 1):
            kind = "X" if (r + c) % 2 == 0 else "Z"
            nb = [(r + a, c + b) for a in (-1, 0) for b in (-1, 0)]
            nb = [(x, y) for (x, y) in nb if 0 <= x < d and 0 <= y < d]
            if len(nb) == 4:
                keep = True
            elif len(nb) == 2:
                on_lr = c == 0 or c == d
                on_tb = r == 0 or r == d
                keep = (kind == "X" and on_lr and not on_tb) or (kind == "Z" and on_tb and not on_lr)
            else:
                keep = False
            if keep:
                out.append((kind, r, c, [x * d + y for (x, y) in nb]))
    xs = [a for a in out if a[0] == "X"]
    zs = [a for a in out if a[0] == "Z"]
    return xs, zs


def check_matrices(d):
    """(H_X, H_Z): [K][d^2] uint8 parity-check matrices in the compact order."""
    xs, zs = ancillas(d)
    hx = np.zeros((len(xs), d * d), dtype=np.uint8)
    hz = np.zeros((len(zs), d * d), dtype=np.uint8)
    for n, a in enumerate(xs):
        hx[n, a[3]] = 1
    for n, a in enumerate(zs):
        hz[n, a[3]] = 1
    return hx, hz


# ---------------------------------------------------------------------------
# Phenomenological noise and detector events
# ---------------------------------------------------------------------------

def sample_noise(d, T, B, p, q, seed):
    """Independent flips, drawn in this order from one PCG64 stream:
    e_z, e_x [B][T][d][d] data-qubit Z / X errors introduced in round t;
    m_x, m_z [B][T][K] measurement errors of round t (K = (d^2-1)/2)."""
    rng = np.random.default_rng(seed)
    K = (d * d - 1) // 2
    e_z = rng.random((B, T, d, d)) < p
    e_x = rng.random((B, T, d, d)) < p
    m_x = rng.random((B, T, K)) < q
    m_z = rng.random((B, T, K)) < q
    return dict(e_z=e_z, e_x=e_x, m_x=m_x, m_z=m_z)


def _syndrome(h, err):
    """Parity of err[..., d^2] on each check row of h -> [..., K]."""
    return (err.astype(np.int64) @ h.T.astype(np.int64)) % 2


def detectors_from_noise(d, noise):
    """Detector bits [B][T][d^2-1] (X-type then Z-type per round), from the
    cumulative outcome s(t) = H * (XOR_{t' <= t} e(t')) XOR m(t)."""
    hx, hz = check_matrices(d)
    e_z, e_x = noise["e_z"], noise["e_x"]
    B, T = e_z.shape[:2]
    acc_z = np.bitwise_xor.accumulate(e_z.reshape(B, T, d * d), axis=1)
    acc_x = np.bitwise_xor.accumulate(e_x.reshape(B, T, d * d), axis=1)
    s_x = _syndrome(hx, acc_z) ^ noise["m_x"]  # X checks see Z errors
    s_z = _syndrome(hz, acc_x) ^ noise["m_z"]  # Z checks see X errors
    s = np.concatenate([s_x, s_z], axis=2).astype(np.uint8)
    prev = np.concatenate([np.zeros_like(s[:, :1]), s[:, :-1]], axis=1)
    return s ^ prev


def ground_truth_flips(d, noise):
    """The flip bits [B][T][3d^2-1] that undo the sampled noise exactly:
    Z data errors, X data errors, X measurement errors, Z measurement errors."""
    e_z, e_x = noise["e_z"], noise["e_x"]
    B, T = e_z.shape[:2]
    return np.concatenate([e_z.reshape(B, T, d * d), e_x.reshape(B, T, d * d),
                           noise["m_x"], noise["m_z"]], axis=2).astype(np.uint8)


# ---------------------------------------------------------------------------
# Packing (LSB-first, whole 64-bit words per sample row)
# ---------------------------------------------------------------------------

def pack_rows(bits):
    """bits [B][n] (0/1) -> [B][ceil(n/64)] uint64, bit b in word b>>6 at position b&63."""
    bits = np.asarray(bits, dtype=np.uint8)
    B, n = bits.shape
    W = (n + 63) // 64
    padded = np.zeros((B, W * 64), dtype=np.uint8)
    padded[:, :n] = bits
    by = np.packbits(padded, axis=1, bitorder="little")
    return np.ascontiguousarray(by).view("<u8").reshape(B, W).astype(np.uint64)


def unpack_rows(words, n):
    words = np.ascontiguousarray(np.asarray(words, dtype=np.uint64))
    B = words.shape[0]
    by = words.astype("<u8").view(np.uint8).reshape(B, -1)
    return np.unpackbits(by, axis=1, bitorder="little")[:, :n]


def make_inputs(d, T, B, p, q, seed):
    """(packed detectors [B][W_det], noise dict)."""
    noise = sample_noise(d, T, B, p, q, seed)
    det = detectors_from_noise(d, noise).reshape(B, -1)
    return pack_rows(det), noise


def config_inputs(cfg_id, batch=None):
    c = CONFIGS[cfg_id]
    return make_inputs(c["d"], c["T"], batch or c["batch"], c["p"], c["q"], 2000 + cfg_id)
