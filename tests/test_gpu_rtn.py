"""GPU parity of the RTN family (per-token symmetric round-to-nearest with no
rotation): the HIP path through the C-ABI against the oracle on the same
seeded inputs.  Codes, scales and the residual window bit-exact; attention
within 1e-2 max-abs; sweep MSE within a relative 2^(b-21)."""
import numpy as np
import pytest

import paper_2605_06675_amd as rq
import workloads
from oracle import calib as ocalib
from oracle import fit as ofit
from tests import gpu_helpers as gh
from tests import test_gpu_parity as gp

pytestmark = pytest.mark.gpu

RTN = workloads.RTN


@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
def test_rtn_every_bit_width(dtype):
    # K widths 2..8 and V widths 8..2 across seven kv-heads, two batch rows
    bits = np.array([[[h + 2, 8 - h] for h in range(7)]])
    print(f"rtn every width dtype {dtype}", flush=True)
    kvc, ks, vs, _ = gp._build(RTN, dtype, 7, 4, 160, 0, bits, batch=2)
    units = gp._check_cache(RTN, dtype, kvc, ks, vs, bits, 0, 2, 7, 160)
    gp._check_attention(kvc, units, dtype, 2, 7, 4)


def test_rtn_window_ragged_tail_chunked_appends():
    # appends of 100, 200, 1 and 32 tokens: block flushes out of the window,
    # a ragged quantized tail and a 16-token window
    bits = np.array([[[3, 2], [5, 4]]])
    print("rtn window + chunks", flush=True)
    kvc, ks, vs, _ = gp._build(RTN, workloads.BF16, 2, 8, 333, 16, bits,
                               cap=352, chunks=[100, 200, 1, 32])
    units = gp._check_cache(RTN, workloads.BF16, kvc, ks, vs, bits, 16, 1, 2,
                            333)
    gp._check_attention(kvc, units, workloads.BF16, 1, 2, 8)


def test_rtn_long_context_many_workgroups():
    # 8 kv-heads x 4 query heads, 2 batch rows, 4113 tokens with a 32-token
    # window: several streaming workgroups per unit and their merge
    rng = np.random.default_rng(3)
    bits = rng.integers(2, 7, size=(1, 8, 2))
    print("rtn long context", flush=True)
    kvc, ks, vs, _ = gp._build(RTN, workloads.BF16, 8, 4, 4113, 32, bits,
                               batch=2)
    units = gp._check_cache(RTN, workloads.BF16, kvc, ks, vs, bits, 32, 2, 8,
                            4113)
    gp._check_attention(kvc, units, workloads.BF16, 2, 8, 4)


@pytest.mark.parametrize("bits", [[2, 3, 4, 5, 6], [4, 5, 6, 7, 8]])
def test_rtn_calibration_sweep(bits):
    """8 key + 8 value components x 512 tokens."""
    gp._torch()
    dtype = workloads.F16
    x16 = workloads.calib_cpu(16, 512, dtype)
    x = workloads.u16_to_f32(x16, dtype)
    for is_value, sl in ((0, slice(0, 8)), (1, slice(8, 16))):
        print(f"rtn sweep bits {bits} value {is_value}", flush=True)
        mse, a, b, r2 = rq.rq_calibrate_distortion(
            RTN, dtype, gh.dev(np.ascontiguousarray(x16[sl]), dtype),
            is_value, bits)
        want = ocalib.sweep(RTN, x[sl], bits, bool(is_value))
        tol = np.array([2.0 ** (bb - 21) for bb in bits])
        rel = np.abs(mse / want - 1)
        print(f"  max rel {rel.max():.2e}")
        assert np.all(rel <= tol[None, :])
        wa, wb, _ = ofit.fit_distortion(want, bits)
        np.testing.assert_allclose(a, wa, rtol=1e-4)
        np.testing.assert_allclose(b, wb, rtol=1e-4)
