"""GPU parity of the mixed family (KIVI keys, RTN per-token symmetric
values; Sec. 3.4 treats K and V as separate components, so each side may
take its own base quantizer): the HIP path through the C-ABI against the
oracle on the same seeded inputs.  Codes, metadata (512 bytes per key block,
64 per value block) and the window bit-exact; attention within 1e-2 at unit
scale; the calibration sweep of each side equals that side's family."""
import numpy as np
import pytest

import paper_2605_06675_amd as rq
import workloads
from oracle import calib as ocalib
from tests import gpu_helpers as gh
from tests import test_gpu_parity as gp

pytestmark = pytest.mark.gpu

MIX = workloads.KIVI_RTN


@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
def test_mixed_every_bit_width(dtype):
    # K widths 1..8, V widths 8..2 across eight kv-heads, two batch rows,
    # 200 tokens with a 32-token window (160 quantized, ragged window)
    bits = np.array([[[h + 1, max(2, 8 - h)] for h in range(8)]])
    print(f"mixed every width dtype {dtype}", flush=True)
    kvc, ks, vs, _ = gp._build(MIX, dtype, 8, 4, 200, 32, bits, batch=2,
                               cap=256)
    units = gp._check_cache(MIX, dtype, kvc, ks, vs, bits, 32, 2, 8, 200)
    gp._check_attention(kvc, units, dtype, 2, 8, 4)


def test_mixed_window_ragged_tail_chunked_appends():
    # appends of 100, 200, 1 and 32 tokens: block flushes out of a 16-token
    # window and a ragged quantized tail
    bits = np.array([[[1, 2], [3, 4]]])
    print("mixed window + chunks", flush=True)
    kvc, ks, vs, _ = gp._build(MIX, workloads.BF16, 2, 8, 333, 16, bits,
                               cap=352, chunks=[100, 200, 1, 32])
    units = gp._check_cache(MIX, workloads.BF16, kvc, ks, vs, bits, 16, 1, 2,
                            333)
    gp._check_attention(kvc, units, workloads.BF16, 1, 2, 8)


@pytest.mark.parametrize("G", [1, 3, 6])
def test_mixed_long_context_group_sizes(G):
    # 4113 tokens: several streaming workgroups per unit and their merge;
    # group sizes that are not powers of two leave query rows unused
    rng = np.random.default_rng(5)
    H = 4
    bits = np.stack([rng.integers(1, 5, size=(1, H)),
                     rng.integers(2, 5, size=(1, H))], axis=-1)
    print(f"mixed long context G {G}", flush=True)
    kvc, ks, vs, _ = gp._build(MIX, workloads.BF16, H, G, 4113, 32, bits,
                               batch=2)
    units = gp._check_cache(MIX, workloads.BF16, kvc, ks, vs, bits, 32, 2, H,
                            4113)
    gp._check_attention(kvc, units, workloads.BF16, 2, H, G)


def test_mixed_calibration_sweep_per_side():
    """4 key + 4 value components x 256 tokens: the mixed family's sweep
    of keys is KIVI's and of values RTN's."""
    gp._torch()
    dtype = workloads.F16
    bits = [2, 3, 4, 5]
    x16 = workloads.calib_cpu(8, 256, dtype)
    x = workloads.u16_to_f32(x16, dtype)
    for is_value, sl, base in ((0, slice(0, 4), workloads.KIVI),
                               (1, slice(4, 8), workloads.RTN)):
        print(f"mixed sweep value {is_value}", flush=True)
        xd = gh.dev(np.ascontiguousarray(x16[sl]), dtype)
        mse, _, _, _ = rq.rq_calibrate_distortion(MIX, dtype, xd, is_value,
                                                  bits)
        same, _, _, _ = rq.rq_calibrate_distortion(base, dtype, xd, is_value,
                                                   bits)
        np.testing.assert_array_equal(mse, same)
        want = ocalib.sweep(MIX, x[sl], bits, bool(is_value))
        rel = np.abs(mse / want - 1)
        tol = np.array([2.0 ** (bb - 21) for bb in bits])
        assert np.all(rel <= tol[None, :]), rel.max()


def test_mixed_rejects_one_bit_values():
    bits = np.array([[[2, 1]]])
    with pytest.raises(rq.RQError):
        rq.KVCache(MIX, workloads.BF16, 1, 1, 1, 4, 64, 0, bits)
