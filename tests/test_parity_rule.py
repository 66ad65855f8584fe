"""The parity rule of tests/parity.py can fail (CPU, oracle outputs only):
a flip or residual bit changed at a site outside the excuse band is counted
as a mismatch and rejected, one inside it is counted as excused; the band
comes from the oracle's logits and the stated tolerance alone; and
assert_flips_follow_logits rejects flips that do not follow the logits."""
import numpy as np
import pytest

import oracle
from fp8_cases import FP8_CASES, case_inputs
from paper_2604_12841_amd import workload
from parity import TOL, assert_flips_follow_logits, assert_parity, compare, flip_sites


def _fp8_reference():
    d, T, layers, weights, det, layout, first, last = case_inputs(FP8_CASES[0])
    ref = oracle.run(d, T, det, layers, weights, bf16=False, layout=layout, first=first, last=last, fp8=True)
    return d, T, det, layout, ref


def _site_logit(d, T, logits, b, bit):
    """Oracle logit of packed flip bit `bit` of sample b."""
    F = 3 * d * d - 1
    t, n = divmod(bit, F)
    ch, i, j = flip_sites(d)[n]
    return logits[b, ch, t, i, j]


def _toggle(words, b, bit):
    w = words.copy()
    w[b, bit >> 6] ^= np.uint64(1) << np.uint64(bit & 63)
    return w


@pytest.mark.parametrize("dtype", ["fp8", "bf16"])
def test_flip_outside_band_fails_inside_is_excused(dtype):
    d, T, det, layout, (logits, flips, res) = _fp8_reference()
    tol = TOL[dtype]
    F = T * (3 * d * d - 1)
    vals = np.array([abs(_site_logit(d, T, logits, 0, k)) for k in range(F)])
    outside = int(np.argmax(vals > tol))
    inside = int(np.argmax(vals <= tol))
    assert vals[outside] > tol and vals[inside] <= tol
    # the GPU side of the comparison: the oracle's own outputs, one bit changed
    st = compare(d, T, dtype, logits, flips, res, _toggle(flips, 0, outside), res, logits.astype(np.float32))
    assert st["flip_mismatch"] == 1
    with pytest.raises(AssertionError):
        assert_parity(st, dtype)
    st = compare(d, T, dtype, logits, flips, res, _toggle(flips, 0, inside), res, logits.astype(np.float32))
    assert st["flip_mismatch"] == 0 and st["flip_excused_mismatch"] == 1
    assert_parity(st, dtype)


def test_residual_bit_outside_band_fails():
    d, T, det, layout, (logits, flips, res) = _fp8_reference()
    st = compare(d, T, "fp8", logits, flips, res, flips, res, logits.astype(np.float32))
    assert st["res_mismatch"] == 0 and st["res_excused"] < st["bits"]
    # a residual bit with no excused flip around it
    S = T * (d * d - 1)
    from parity import excused_masks
    _, rex = excused_masks(d, T, logits, TOL["fp8"])
    bit = int(np.argmax(~rex[0]))
    st = compare(d, T, "fp8", logits, flips, res, flips, _toggle(res, 0, bit), logits.astype(np.float32))
    assert st["res_mismatch"] == 1
    with pytest.raises(AssertionError):
        assert_parity(st, "fp8")


def test_excuse_band_does_not_depend_on_the_gpu_logits():
    """The same flips compared with very different 'GPU' logits excuse the
    same sites (the band is the oracle's |logit| <= tol)."""
    d, T, det, layout, (logits, flips, res) = _fp8_reference()
    a = compare(d, T, "fp8", logits, flips, res, flips, res, logits.astype(np.float32))
    b = compare(d, T, "fp8", logits, flips, res, flips, res, (logits + 5.0).astype(np.float32))
    assert a["flip_excused"] == b["flip_excused"] and a["res_excused"] == b["res_excused"]
    assert b["max_abs_logit_err"] > TOL["fp8"]
    with pytest.raises(AssertionError):
        assert_parity(b, "fp8")


def test_logit_bound_is_enforced():
    d, T, det, layout, (logits, flips, res) = _fp8_reference()
    bumped = logits.copy()
    bumped[0, 0, 0, 0, 0] += 1.5 * TOL["bf16"]
    st = compare(d, T, "bf16", logits, flips, res, flips, res, bumped.astype(np.float32))
    with pytest.raises(AssertionError):
        assert_parity(st, "bf16")


def test_flips_follow_logits_detects_a_changed_bit():
    d = T = 5
    layers = workload.layer_spec(2, 8)
    weights = workload.he_normal_weights(layers, seed=70)
    det, _ = workload.make_inputs(d, T, 2, 0.05, 0.05, 71)
    logits, flips, res = oracle.run(d, T, det, layers, weights, bf16=True)
    assert_flips_follow_logits(d, T, det, logits.astype(np.float32), flips, res)
    with pytest.raises(AssertionError):
        assert_flips_follow_logits(d, T, det, logits.astype(np.float32), _toggle(flips, 1, 7), res)
    with pytest.raises(AssertionError):
        assert_flips_follow_logits(d, T, det, logits.astype(np.float32), flips, _toggle(res, 0, 3))
