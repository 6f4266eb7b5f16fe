"""Pins of the decode-attention and distortion-sweep oracles."""
import math

import numpy as np
import pytest
import torch

import workloads
from oracle import attention, cache, calib, fit


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def test_single_token_returns_its_value():
    v = _rand((1, 128), 1)
    out = attention.decode_attention(_rand((4, 128), 2), _rand((1, 128), 3), v)
    np.testing.assert_allclose(out, np.repeat(v, 4, 0), rtol=0, atol=1e-15)


def test_constant_values():
    vrow = _rand((128,), 4)
    v = np.tile(vrow, (50, 1))
    out = attention.decode_attention(_rand((4, 128), 5), _rand((50, 128), 6), v)
    np.testing.assert_allclose(out, np.tile(vrow, (4, 1)), atol=1e-14)


def test_zero_query_gives_mean_value():
    v = _rand((77, 128), 7)
    out = attention.decode_attention(np.zeros((2, 128)), _rand((77, 128), 8), v)
    np.testing.assert_allclose(out, np.tile(v.mean(0), (2, 1)), atol=1e-14)


def test_identical_queries_identical_outputs():
    q = np.tile(_rand((1, 128), 9), (4, 1))
    out = attention.decode_attention(q, _rand((33, 128), 10),
                                     _rand((33, 128), 11))
    assert np.all(out == out[0])


def test_matches_library_sdpa():
    q, k, v = _rand((4, 128), 12), _rand((300, 128), 13), _rand((300, 128), 14)
    want = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, :, None, :],
        torch.from_numpy(k)[None, None].expand(1, 4, 300, 128),
        torch.from_numpy(v)[None, None].expand(1, 4, 300, 128))[0, :, 0]
    np.testing.assert_allclose(attention.decode_attention(q, k, v),
                               want.numpy(), atol=1e-12)


def test_high_bit_cache_close_to_exact():
    # At 8 bits the quantized cache barely changes attention.
    wl = workloads.SMALL
    k16, v16 = workloads.kv_cpu(wl, 0, 0, 512)
    k = workloads.u16_to_f32(k16[0], wl.dtype)
    v = workloads.u16_to_f32(v16[0], wl.dtype)
    q = workloads.u16_to_f32(workloads.q_cpu(wl, 0)[0, :4], wl.dtype)
    u = cache.Unit(cache.KIVI, k, v, 8, 8, 32)
    exact = attention.decode_attention(q, k, v)
    approx = attention.decode_attention(q, u.keys(), u.values())
    assert np.max(np.abs(exact - approx)) < 2e-2
    u2 = cache.Unit(cache.KIVI, k, v, 2, 2, 32)
    low = attention.decode_attention(q, u2.keys(), u2.values())
    assert np.max(np.abs(exact - low)) > np.max(np.abs(exact - approx))


@pytest.mark.parametrize("family", [calib.KIVI, calib.QUAROT])
def test_sweep_monotone_and_fit(family):
    bits = [2, 3, 4, 5, 6]
    x = workloads.u16_to_f32(workloads.calib_cpu(4, 128, workloads.BF16),
                             workloads.BF16)
    for is_value in (False, True):
        D = calib.sweep(family, x, bits, is_value)
        assert np.all(np.diff(D, axis=1) < 0)
        a, b, r2 = fit.fit_distortion(D, bits)
        # a uniform scalar quantizer's MSE falls about 4x per extra bit at
        # high rate, so the fitted beta sits near 4
        assert np.all((b > 3.0) & (b < 5.5)) and np.all(r2 > 0.98)


def test_sweep_lossless_is_zero():
    rng = np.random.default_rng(3)
    # values 0..3 in every group of 32 are exact at 2 bits (s = 1, z = 0)
    k = rng.integers(0, 4, size=(2, 64, 128)).astype(np.float32)
    k[..., ::32] = 0
    k[..., 1::32] = 3
    D = calib.sweep(calib.KIVI, k, [2, 3], is_value=True)
    assert np.all(D[:, 0] == 0) and np.all(D[:, 1] > 0)
