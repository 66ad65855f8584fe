"""Comparison of the GPU path with the CPU oracle (test helper).

Parity rule: logits agree to a max abs error <= tol (2e-2 for bf16, 1e-4 for
fp32, the fp8 bound below for fp8); thresholded flips and residual bits agree
exactly, except at sites whose oracle |logit| <= tol ("excused": there the
two logits may have different signs without breaking the logit bound).  A
residual bit is excused when any of the flips it XORs in is.  Excused counts
are reported; non-excused mismatches must be 0.  The excuse depends on the
oracle's logits and the stated tolerance only, never on the GPU's output.

fp8 (whole networks): the fp8 matrix instruction sums its products with an
error up to about 2^-16 of their magnitudes, so an activation next to an
E4M3 rounding boundary can round either way, and the difference (one E4M3
step) spreads through the later layers.  The max abs logit error is bounded
by tests/golden/make_fp8_tolerance.py from the oracle alone (its fp8 forward
with every sum moved by up to that error, over several hashed patterns,
times a margin), and the same bound sets the excused sites.  Tight per-site
checks of the fp8 layers are in test_gpu_fp8.py.

assert_flips_follow_logits checks the GPU's threshold, bit packing and
residual on its own logits, with nothing excused.
"""
import functools
import json
import os

import numpy as np

import oracle
from paper_2604_12841_amd import workload

_FP8 = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "fp8_tolerance.json")))
TOL = {"bf16": 2e-2, "fp32": 1e-4, "fp8": _FP8["tol_max_abs_logit_err"]}
FAR_ABS = 1e-3  # a logit "far" from the oracle's (reported)


@functools.lru_cache(maxsize=None)
def flip_sites(d, layout="plaquette"):
    """(ch, i, j) of each compact flip index n in [0, 3d^2 - 1): where its
    logit sits on the grid of the layout."""
    site_of, _ = oracle.stabilizer_order(d)
    H = d + 1
    K = (d * d - 1) // 2
    out = [(0, r, c) for r in range(d) for c in range(d)]
    out += [(1, r, c) for r in range(d) for c in range(d)]
    for n in range(d * d - 1):
        i, j = divmod(int(site_of[n]), H)
        if layout == "paper":
            _, i, j = oracle.stabilizer_qubit(d, i, j)
        out.append((2 if n < K else 3, i, j))
    return np.array(out, dtype=np.int64)


@functools.lru_cache(maxsize=None)
def residual_contributions(d):
    """For each stabilizer n: (flip index of its measurement correction,
    list of flip indices of the data corrections on its support)."""
    site_of, _ = oracle.stabilizer_order(d)
    H = d + 1
    K = (d * d - 1) // 2
    meas, data = [], []
    for n in range(d * d - 1):
        i, j = divmod(int(site_of[n]), H)
        meas.append(2 * d * d + n)
        ch = 0 if n < K else 1
        sup = [ch * d * d + r * d + c for (r, c) in oracle.plaquette_support(d, i, j)]
        data.append(sup + [-1] * (4 - len(sup)))
    return np.array(meas), np.array(data)


def excused_masks(d, T, logits, tol, layout="plaquette"):
    """(flip_excused [B][T*(3d^2-1)], residual_excused [B][T*(d^2-1)]) bool:
    flips whose oracle |logit| <= tol, and the residual bits they reach."""
    fs = flip_sites(d, layout)
    B = logits.shape[0]
    F = 3 * d * d - 1
    S = d * d - 1
    sel = (slice(None), fs[:, 0][None, :].repeat(T, 0), np.arange(T)[:, None], fs[:, 1][None, :], fs[:, 2][None, :])
    lf = logits[sel]
    fex = (np.abs(lf) <= tol).reshape(B, T, F)
    meas, data = residual_contributions(d)
    rex = fex[:, :, meas].copy()
    rex[:, 1:] |= fex[:, :-1, meas]
    for q in range(4):
        idx = data[:, q]
        ok = idx >= 0
        part = np.zeros((B, T, S), dtype=bool)
        part[:, :, ok] = fex[:, :, idx[ok]]
        rex |= part
    return fex.reshape(B, T * F), rex.reshape(B, T * S)


def compare(d, T, dtype, ref_logits, ref_flips, ref_res, got_flips, got_res, got_logits=None,
            layout="plaquette", tol=None):
    """Returns a dict of parity statistics (see module docstring); tol
    defaults to the dtype's logit tolerance."""
    tol = TOL[dtype] if tol is None else tol
    B = ref_logits.shape[0]
    F = T * (3 * d * d - 1)
    S = T * (d * d - 1)
    err = None if got_logits is None else np.abs(got_logits.astype(np.float64) - ref_logits)
    fex, rex = excused_masks(d, T, ref_logits, tol, layout)
    rf = workload.unpack_rows(ref_flips, F).astype(bool)
    gf = workload.unpack_rows(got_flips, F).astype(bool)
    rr = workload.unpack_rows(ref_res, S).astype(bool)
    gr = workload.unpack_rows(got_res, S).astype(bool)
    out = dict(
        flip_mismatch=int(((rf != gf) & ~fex).sum()),
        flip_excused=int(fex.sum()),
        flip_excused_mismatch=int(((rf != gf) & fex).sum()),
        res_mismatch=int(((rr != gr) & ~rex).sum()),
        res_excused=int(rex.sum()),
        flips_set=int(rf.sum()),
        residual_set=int(rr.sum()),
        bits=B * (F + S),
        # padding bits beyond the last flip / residual bit must be zero
        flip_padding_ok=bool(_padding_zero(got_flips, F)),
        res_padding_ok=bool(_padding_zero(got_res, S)),
    )
    if err is not None:
        out["max_abs_logit_err"] = float(err.max())
        out["frac_far"] = float((err > FAR_ABS).mean())
    return out


def assert_flips_follow_logits(d, T, det, got_logits, got_flips, got_res, layout="plaquette"):
    """The GPU's packed flips and residual equal the oracle's threshold,
    packing and residual applied to the GPU's own logits (exactly)."""
    f = oracle.flips_residual_paper if layout == "paper" else oracle.flips_residual
    flips, res = f(d, T, np.asarray(got_logits, dtype=np.float64), det)
    np.testing.assert_array_equal(np.asarray(got_flips, dtype=np.uint64), flips)
    np.testing.assert_array_equal(np.asarray(got_res, dtype=np.uint64), res)


def _padding_zero(words, nbits):
    words = np.asarray(words, dtype=np.uint64)
    rem = nbits % 64
    if rem == 0:
        return True
    return bool((words[:, -1] >> np.uint64(rem) == 0).all())


def assert_parity(stats, dtype, tol=None):
    tol = TOL[dtype] if tol is None else tol
    assert stats["flip_padding_ok"] and stats["res_padding_ok"], stats
    assert stats["flip_mismatch"] == 0, stats
    assert stats["res_mismatch"] == 0, stats
    if "max_abs_logit_err" in stats:
        assert stats["max_abs_logit_err"] <= tol, stats


def config_case(cfg_id, batch=None, act=workload.GELU_TANH):
    c = workload.CONFIGS[cfg_id]
    layers = workload.config_layers(cfg_id, act)
    weights = workload.config_weights(cfg_id, act)
    det, noise = workload.config_inputs(cfg_id, batch)
    return c["d"], c["T"], c["dtype"], layers, weights, det, noise


# ---- GPU-side helpers shared by the GPU tests (torch is imported lazily so
# the CPU suite does not need a device) ----

def say(*a):
    import sys
    print(*a, file=sys.stderr, flush=True)


def dev_u64(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint64).view(np.int64)).cuda()


def host_u64(t):
    return t.cpu().numpy().view(np.uint64)


def run_gpu(pre, det, want_logits=True, canary=True, batch=None):
    """One predecoder_run of the first `batch` rows of det (default: all) into
    freshly filled outputs (-1 / NaN canaries); returns host arrays."""
    import torch
    B = det.shape[0] if batch is None else batch
    d, T = pre.d, pre.T
    ddet = dev_u64(det[:B])
    fill = -1 if canary else 0
    flips = torch.full((B, pre.flip_words), fill, dtype=torch.int64, device="cuda")
    res = torch.full((B, pre.det_words), fill, dtype=torch.int64, device="cuda")
    logits = None
    if want_logits:
        logits = torch.full((B, 4, T, pre.grid, pre.grid), float("nan"), dtype=torch.float32, device="cuda")
    pre.run(ddet, flips, res, logits)
    torch.cuda.synchronize()
    return host_u64(flips), host_u64(res), (logits.cpu().numpy() if want_logits else None)
