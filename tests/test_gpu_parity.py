"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Every case prints its name, seed and shape before touching the GPU.  The
oracle and the GPU consume the same seeded arrays from the workload module.
"""
import numpy as np
import pytest

import oracle
import paper_2604_12841_amd as pdx
from paper_2604_12841_amd import workload
from parity import assert_parity, compare, config_case, dev_u64, host_u64, run_gpu, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cuda():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda")


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_unpack_bit_exact(cuda, cfg):
    d, T, dtype, layers, weights, det, _ = config_case(cfg, batch=3)
    say("unpack cfg", cfg, "d", d, "T", T, "B", 3)
    pre = pdx.Predecoder(weights, d, T, layers, dtype, max_batch=3)
    H = d + 1
    tdt = torch.float32 if dtype == "fp32" else torch.int16
    planes = torch.full((3, T, H, H, 2), -1, dtype=tdt, device="cuda")
    pre.unpack(dev_u64(det), planes)
    torch.cuda.synchronize()
    got = planes.cpu().numpy()
    if dtype == "bf16":
        got = got.view(np.uint16)
        assert set(np.unique(got).tolist()) <= {0, 0x3F80}
        got = (got == 0x3F80).astype(np.float64)
    ref = oracle.unpack(d, T, det).transpose(0, 2, 3, 4, 1)
    np.testing.assert_array_equal(got, ref)
    pre.close()


# (config, batch) small enough for the oracle to finish in seconds
SMALL = [(1, 64), (2, 8), (3, 3), (4, 1), (5, 1)]


@pytest.mark.parametrize("cfg,batch", SMALL)
def test_full_path_parity(cuda, cfg, batch):
    d, T, dtype, layers, weights, det, _ = config_case(cfg, batch=batch)
    say("full path cfg", cfg, "d", d, "T", T, "B", batch, "dtype", dtype)
    pre = pdx.Predecoder(weights, d, T, layers, dtype, max_batch=batch)
    flips, res, logits = run_gpu(pre, det)
    ref_logits, ref_flips, ref_res = oracle.run(d, T, det, layers, weights, bf16=(dtype == "bf16"))
    st = compare(d, T, dtype, ref_logits, ref_flips, ref_res, flips, res, logits)
    say("  stats", st)
    assert_parity(st, dtype)
    pre.close()


def test_ground_truth_flips_zero_residual(cuda):
    for cfg in (1, 3, 5):
        d, T, dtype, layers, weights, det, noise = config_case(cfg, batch=4)
        say("residual from ground-truth flips cfg", cfg)
        pre = pdx.Predecoder(weights, d, T, layers, dtype, max_batch=4)
        gt = workload.pack_rows(workload.ground_truth_flips(d, noise).reshape(4, -1))
        res = torch.full((4, pre.det_words), -1, dtype=torch.int64, device="cuda")
        pre.residual(dev_u64(det), dev_u64(gt), res)
        torch.cuda.synchronize()
        assert not host_u64(res).any()
        # arbitrary flips: the GPU residual stage equals the oracle's
        rng = np.random.default_rng(cfg)
        fl = workload.pack_rows((rng.random((4, T * (3 * d * d - 1))) < 0.05).astype(np.uint8))
        pre.residual(dev_u64(det), dev_u64(fl), res)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host_u64(res), oracle.residual_from_flips(d, T, det, fl))
        pre.close()


def test_deterministic(cuda):
    d, T, dtype, layers, weights, det, _ = config_case(3, batch=16)
    say("determinism cfg 3 B 16")
    pre = pdx.Predecoder(weights, d, T, layers, dtype, max_batch=16)
    a = run_gpu(pre, det)
    b = run_gpu(pre, det)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    pre.close()
