"""Tight checks of the activations a GPU layer stores (test helper).

Each check recomputes one layer in fp64 from the GPU's own input (the planes
for the first layer, else what the GPU stored for the layer before), with the
precision points of the handle: weights as the library uses them, the sum of
products, the bias (and a residual block's shortcut), the activation, then
rounding to the stored format (bf16 round-to-nearest-even, or E4M3 through
PyTorch's float8_e4m3fn, which the oracle's encoder is pinned against).

The GPU sums its products in fp32 (and, for fp8, inside a matrix instruction
whose own sum is not exact), so its pre-activation may differ from the fp64
value by up to a bound eps_abs; its activation arithmetic adds a relative
error of at most act_rel_err (GELU as y / (1 + 2^z), z = y (c1 + c3 y^2): a
few fp32 roundings in z, which exp2 turns into a relative error of about
|z| ln 2 times theirs, plus the exp2, the addition, the reciprocal and the
product; ReLU and no activation are exact).  Every stored value
must then be the exact rounding of the fp64 result, except where the window
[y - eps_abs, y + eps_abs] (and the activation error) reaches a rounding
boundary: there it must be one of the values reachable inside the window.
Anything else -- a wrong tap, channel, bias, shortcut or rounding -- moves
values by whole steps of the stored format and fails.

Sum bounds (per output value, relative to the sum of the magnitudes of its
products plus |bias|):
* bf16 matrix instructions (v_mfma_f32_32x32x16_bf16): 16 exact products per
  instruction, accumulated in fp32; over K products a chain of K/16
  instruction steps, each adding one rounding of at most 2^-24 of the running
  magnitude, plus the instruction's own 16-term sum (taken as up to four
  more roundings): (ceil(K / 16) + 4) 2^-24.
* fp32 FMA chains (the projection shortcut, K terms): (K + 1) 2^-24.
* fp8 matrix instructions: measured on gfx950 at about 2^-16.4 per sum of 64
  products (reading 18 of the design notes), taken as 2^-16 + 2^-18; the
  first layer (bf16 instructions over the dequantised weights) 2^-17.
"""
import numpy as np
import torch

F = torch.nn.functional

U32 = 2.0 ** -24
GELU_MIN_AT = -0.7517  # GELU-tanh is not monotonic around its minimum
GELU_C1 = 2.0 * np.log2(np.e) * np.sqrt(2.0 / np.pi)
GELU_C3 = GELU_C1 * 0.044715

NONE, GELU_TANH, RELU = 0, 1, 2


def eps_bf16_mfma(k_terms):
    return (int(np.ceil(k_terms / 16)) + 4) * U32


def eps_fma_chain(k_terms):
    return (k_terms + 1) * U32


def q_bf16(t):
    return t.float().to(torch.bfloat16).double()


def q_e4m3(t):
    return t.float().clamp(-448.0, 448.0).to(torch.float8_e4m3fn).double()


def act_fn(v, act):
    """The activation in fp64 of the fp32-rounded input, rounded to fp32.
    GELU (tanh form) as y / (1 + exp(-2u)), the same function as 0.5 y (1 +
    tanh(u)) without that form's cancellation at large negative y (the
    oracle's evaluation, pinned against a 160-digit one)."""
    v = v.float().double()
    if act == GELU_TANH:
        u = np.sqrt(2.0 / np.pi) * (v + 0.044715 * v ** 3)
        v = v / (1.0 + torch.exp(-2.0 * u))
    elif act == RELU:
        v = F.relu(v)
    return v.float().double()


def act_rel_err(y, act):
    """Bound on the relative error of the GPU's activation at pre-activation y."""
    if act != GELU_TANH:
        return torch.zeros_like(y)
    z = (y.abs() + 1.0) * (GELU_C1 + GELU_C3 * (y.abs() + 1.0) ** 2)
    return (8.0 + 3.0 * z) * U32


def expected(y, eps_abs, act, quant):
    """The exact stored value of pre-activations y, and the lowest and
    highest stored values reachable when y moves by up to eps_abs and the
    activation by up to act_rel_err (rounding is monotone, and so is the
    activation on either side of GELU's minimum, whose value is included
    when the window contains it); every representable value in between is
    reachable too."""
    exact = quant(act_fn(y, act))
    rel = act_rel_err(y.abs() + eps_abs, act)
    lo, hi = exact.clone(), exact.clone()
    for dy in (-1.0, -0.5, 0.5, 1.0):
        for r in (-1.0, 1.0):
            c = quant(act_fn(y + dy * eps_abs, act) * (1.0 + r * rel))
            lo = torch.minimum(lo, c)
            hi = torch.maximum(hi, c)
    if act == GELU_TANH:
        spans_min = (y - eps_abs < GELU_MIN_AT) & (y + eps_abs > GELU_MIN_AT)
        vmin = quant(act_fn(torch.full_like(y, GELU_MIN_AT), act) * (1.0 + rel))
        lo = torch.where(spans_min, torch.minimum(lo, vmin), lo)
    return exact, lo, hi


def check_stored(name, got, y, eps_abs, act, quant, say=print):
    """Asserts the rule above for stored values `got` (fp64 tensor of the
    stored values) against pre-activations y; returns counts."""
    exact, lo, hi = expected(y, eps_abs, act, quant)
    amb = lo != hi
    exact_bad = int(((got != exact) & ~amb).sum())
    window_bad = int((((got < lo) | (got > hi)) & amb).sum())
    st = dict(values=got.numel(), ambiguous=int(amb.sum()), differ_in_window=int(((got != exact) & amb).sum()),
              exact_bad=exact_bad, window_bad=window_bad)
    say("  %s: values %d, in a window %d (%.4f), differing there %d, mismatches %d + %d" %
        (name, st["values"], st["ambiguous"], st["ambiguous"] / max(1, st["values"]), st["differ_in_window"],
         exact_bad, window_bad))
    if exact_bad or window_bad:
        bad = (((got != exact) & ~amb) | (((got < lo) | (got > hi)) & amb)).nonzero()
        for idx in bad[:8].tolist():
            idx = tuple(idx)
            say("    at %s: y %.9g eps %.3g stored %.9g exact %.9g window [%.9g, %.9g]" %
                (idx, float(y[idx]), float(eps_abs[idx]), float(got[idx]), float(exact[idx]), float(lo[idx]),
                 float(hi[idx])))
    assert exact_bad == 0 and window_bad == 0, (name, st)
    return st


def conv(x, w, b=None, k=3):
    return F.conv3d(x, w, b, padding=(k - 1) // 2)


def conv_mag(x, w, b=None, k=3):
    """Sum of the magnitudes of each output's products, plus |bias|."""
    m = F.conv3d(x.abs(), w.abs(), None, padding=(k - 1) // 2)
    if b is not None:
        m = m + b.abs().reshape(1, -1, 1, 1, 1)
    return m


def bf16_bits_to_double(t):
    """[..] int16 tensor of bf16 bit patterns -> fp64 values."""
    return (t.to(torch.int32) << 16).view(torch.float32).double()
