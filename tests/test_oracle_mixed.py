"""Oracle of the mixed family (KIVI-style per-channel asymmetric keys with
RTN per-token symmetric values: each side its own base quantizer, which the
paper's K/V separation allows, Sec. 3.4).  Pinned by reduction: every key
code, scale and zero point equals the KIVI family's for the same inputs,
every value code and scale equals the RTN family's, and so do the
dequantized caches, the distortion sweeps and decode attention."""
import numpy as np
import pytest

import workloads
from oracle import attention as oatt
from oracle import cache as ocache
from oracle import calib as ocalib

T, R = 200, 32


def _kv(seed):
    wl = workloads.Workload("t", ocache.KIVI_RTN, workloads.BF16, 1, 1, 4, 16, T, R,
                            (1,), 2.0, 0.5, (1.0, 1.0))
    k16, v16 = workloads.kv_cpu(wl, 0, 0, T, seed=seed)
    return (workloads.u16_to_f32(k16, workloads.BF16),
            workloads.u16_to_f32(v16, workloads.BF16))


@pytest.mark.parametrize("bk,bv", [(1, 2), (2, 3), (3, 4), (4, 8), (8, 2)])
def test_mixed_unit_is_kivi_keys_and_rtn_values(bk, bv):
    k, v = _kv(3)
    for h in range(k.shape[0]):
        m = ocache.Unit(ocache.KIVI_RTN, k[h], v[h], bk, bv, R)
        a = ocache.Unit(ocache.KIVI, k[h], v[h], bk, 2, R)
        r = ocache.Unit(ocache.RTN, k[h], v[h], 2, bv, R)
        np.testing.assert_array_equal(m.k_codes, a.k_codes)
        np.testing.assert_array_equal(m.k_words, a.k_words)
        np.testing.assert_array_equal(np.asarray(m.k_meta).view(np.uint16),
                                      np.asarray(a.k_meta).view(np.uint16))
        np.testing.assert_array_equal(m.v_codes, r.v_codes)
        np.testing.assert_array_equal(m.v_words, r.v_words)
        np.testing.assert_array_equal(np.asarray(m.v_meta).view(np.uint16),
                                      np.asarray(r.v_meta).view(np.uint16))
        np.testing.assert_array_equal(m.keys(), a.keys())
        np.testing.assert_array_equal(m.values(), r.values())
        q = np.random.default_rng(h).standard_normal((4, 128))
        np.testing.assert_allclose(oatt.decode_attention(q, m.keys(), m.values()),
                                   oatt.decode_attention(q, a.keys(), r.values()),
                                   rtol=0, atol=0)


def test_mixed_sweep_is_kivi_for_keys_and_rtn_for_values():
    k, v = _kv(5)
    k, v = k[:, :192], v[:, :192]       # whole 32-token groups
    bits = [2, 3, 4]
    np.testing.assert_array_equal(ocalib.sweep(ocache.KIVI_RTN, k, bits, False),
                                  ocalib.sweep(ocache.KIVI, k, bits, False))
    np.testing.assert_array_equal(ocalib.sweep(ocache.KIVI_RTN, v, bits, True),
                                  ocalib.sweep(ocache.RTN, v, bits, True))
