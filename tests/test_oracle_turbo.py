"""Pins of the TurboQuant-style quantizer oracle (rotation + Lloyd-Max
codebook of N(0,1); Sec. 2, Sec. 3.1 and its Table 6)."""
import math

import numpy as np
import pytest

import workloads
from oracle import cache, calib, fit, quant
from tests.golden import load as golden

T6 = golden.table("table6_lloydmax.txt")


def _rot(seed=42, layer=0, head=0):
    r16 = workloads.turbo_rotation(seed, layer, head)
    return workloads.u16_to_f32(r16, workloads.BF16).astype(np.float64)


def test_rotation_is_orthogonal_to_bf16_precision():
    for s in range(6):
        R = _rot(s, s % 3, s % 5)
        # bf16 keeps 8 significant bits: each entry is within 2^-9 relative
        assert np.abs(R @ R.T - np.eye(128)).max() < 2.0 ** -8
    assert np.array_equal(workloads.turbo_rotation(1, 2, 3),
                          workloads.turbo_rotation(1, 2, 3))
    assert not np.array_equal(workloads.turbo_rotation(1, 2, 3),
                              workloads.turbo_rotation(1, 2, 4))


@pytest.mark.parametrize("b", [1, 2, 3, 4])
def test_identity_rotation_is_scalar_lloyd_max(b):
    # With R = I and |x| = sqrt(128), t = x up to the fp16 rounding of the
    # norm: each coordinate gets the nearest Lloyd-Max centroid (midpoint
    # thresholds), found by brute force.
    rng = np.random.default_rng(b)
    x = rng.standard_normal((40, 128))
    x = x / np.linalg.norm(x, axis=1, keepdims=True) * math.sqrt(128)
    x = x.astype(np.float32)
    u, n, t = quant.turbo_quant(x, np.eye(128), b)
    np.testing.assert_allclose(t, x, rtol=2.0 ** -10)
    c, _ = quant.turbo_codebook(b)
    want = np.argmin(np.abs(t[..., None] - c), axis=-1)
    assert np.array_equal(u, want)


def test_codes_count_thresholds_below():
    th = quant.turbo_codebook(3)[1].astype(np.float64)
    # a vector whose rotated, normalised coordinates sit between thresholds
    t = np.concatenate([th - 1e-3, th + 1e-3, [-9.0, 9.0]])
    t = np.resize(t, 128)
    x = (t / math.sqrt(128)).astype(np.float32)
    u, n, tt = quant.turbo_quant(x[None], np.eye(128), 3)
    want = np.array([np.sum(v > th) for v in tt[0]])
    assert np.array_equal(u[0], want)
    assert u.min() == 0 and u.max() == 7


@pytest.mark.parametrize("b", [2, 3, 4])
def test_sign_symmetry(b):
    R = _rot()
    x = np.random.default_rng(7).standard_normal((16, 128)).astype(np.float32)
    u, _, t = quant.turbo_quant(x, R, b)
    um, _, tm = quant.turbo_quant(-x, R, b)
    assert np.allclose(tm, -t)
    off = ~quant.turbo_near_threshold(t, b, 1e-12)
    assert np.array_equal(um[off], (1 << b) - 1 - u[off])


def test_zero_vector_and_power_of_two_scale():
    R = _rot()
    for b in (1, 3):
        u, n, _ = quant.turbo_quant(np.zeros((1, 128), np.float32), R, b)
        assert n[0] == 0 and np.all(u == (1 << (b - 1)) - 1)
        assert np.all(quant.turbo_dequant(u, n, R, b) == 0)
    x = np.random.default_rng(3).standard_normal((8, 128)).astype(np.float32)
    u1, n1, _ = quant.turbo_quant(x, R, 4)
    u2, n2, _ = quant.turbo_quant(x * np.float32(8), R, 4)
    assert np.array_equal(u1, u2)
    assert np.array_equal(n2.astype(np.float64), 8 * n1.astype(np.float64))


@pytest.mark.parametrize("b", [1, 2, 3, 4])
def test_gaussian_mse_close_to_table6(b):
    # Rotated Gaussian data: each normalised coordinate is close to N(0,1),
    # so the per-element MSE is close to Table 6's Lloyd-Max value (within
    # the O(1/d) and bf16-rotation effects).
    R = _rot(5)
    x = np.random.default_rng(10 + b).standard_normal((2000, 128)).astype(np.float32)
    u, n, _ = quant.turbo_quant(x, R, b)
    xh = quant.turbo_dequant(u, n, R, b)
    mse = np.mean((x.astype(np.float64) - xh) ** 2)
    assert abs(mse / T6[b - 1, 1] - 1) < 0.06


def test_norm_rounding_rule():
    x = np.random.default_rng(4).standard_normal((32, 128)).astype(np.float32)
    n = quant.turbo_norm(x)
    exact = np.sqrt((x.astype(np.float64) ** 2).sum(axis=1))
    assert np.array_equal(n, exact.astype(np.float32).astype(np.float16))
    assert np.all(np.abs(n.astype(np.float64) / exact - 1) <= 2.0 ** -11 * 1.01)


def test_unit_layout_roundtrip():
    R = _rot(9)
    k = np.random.default_rng(1).standard_normal((100, 128)).astype(np.float32)
    v = np.random.default_rng(2).standard_normal((100, 128)).astype(np.float32)
    u = cache.Unit(cache.TURBO, k, v, 3, 2, 0, rotation=R)
    assert u.nq == 96
    assert np.array_equal(cache.unpack_keys(u.k_words, 3), u.k_codes)
    assert np.array_equal(cache.unpack_values(u.v_words, 2), u.v_codes)
    assert u.k_meta.shape == (3, 32) and u.k_meta.dtype == np.float16
    # dequantized keys are close to the inputs at 3 bits
    err = np.mean((u.k_hat - k[:96]) ** 2) / np.mean(k[:96] ** 2)
    assert err < 0.05


def test_sweep_fit_near_lloyd_max_curve():
    # The TurboQuant sweep on Gaussian data follows the Lloyd-Max curve, so
    # the fitted beta is near the 3.48 of Table 6's fit (Sec. 3.1).
    x = np.random.default_rng(0).standard_normal((2, 256, 128)).astype(np.float32)
    rots = np.stack([_rot(1), _rot(2)])
    D = calib.sweep(calib.TURBO, x, [1, 2, 3, 4], False, rots)
    assert np.all(np.diff(D, axis=1) < 0)
    a, b, r2 = fit.fit_distortion(D, [1, 2, 3, 4])
    assert np.all((b > 3.2) & (b < 3.9)) and np.all(r2 > 0.99)
