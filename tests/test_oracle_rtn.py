"""Pins of the RTN oracle (per-token symmetric round-to-nearest, Appendix
"RTN Base Quantizer").

The quantizer's definition fixes: one scale per token with the token's
largest magnitude on the top level (up to the fp16 rounding of the scale),
each element on the nearest of the 2^b - 1 symmetric levels, and exact
reconstruction of values already on the grid.  The tests below check those
facts by brute force and by closed forms, not by re-deriving the formula."""
import numpy as np
import pytest

from oracle import cache, calib, quant

F32 = np.float32


def _tokens(seed, T=48, scale=1.0):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, 128)) * scale
    return x.astype(np.float16).astype(F32)


@pytest.mark.parametrize("b", [2, 3, 4, 5, 8])
def test_codes_are_the_nearest_level_brute_force(b):
    x = _tokens(b)
    u, s = quant.rtn_quant(x, b)
    qm = (1 << (b - 1)) - 1
    assert u.shape == x.shape and s.shape == (x.shape[0],)
    assert u.min() >= 1 and u.max() <= 2 * qm + 1        # codes 1 .. 2^b - 1
    sf = s.astype(np.float64)
    levels = np.arange(-qm, qm + 1, dtype=np.float64)
    checked = 0
    for t in range(x.shape[0]):
        d = np.abs(x[t].astype(np.float64)[:, None] - levels[None, :] * sf[t])
        order = np.sort(d, axis=1)
        clear = order[:, 1] - order[:, 0] > 1e-6 * sf[t]  # no near tie
        best = levels[np.argmin(d, axis=1)].astype(np.int64)
        assert np.array_equal((u[t] - (1 << (b - 1)))[clear], best[clear])
        checked += clear.sum()
    assert checked > 0.99 * x.size


@pytest.mark.parametrize("b", [2, 3, 4, 6])
def test_scale_puts_the_largest_magnitude_on_the_top_level(b):
    x = _tokens(10 + b)
    _, s = quant.rtn_quant(x, b)
    qm = (1 << (b - 1)) - 1
    a = np.max(np.abs(x.astype(np.float64)), axis=1)
    # fp16 keeps 11 significant bits: relative rounding error <= 2^-11
    assert np.all(np.abs(s.astype(np.float64) * qm - a) <= 2.0 ** -11 * a * 1.0001)


@pytest.mark.parametrize("b", [2, 3, 4, 5, 8])
def test_error_bound(b):
    x = _tokens(20 + b)
    u, s = quant.rtn_quant(x, b)
    xh = quant.rtn_dequant(u, s, b)
    qm = (1 << (b - 1)) - 1
    sf = s.astype(np.float64)[:, None]
    a = np.max(np.abs(x.astype(np.float64)), axis=1, keepdims=True)
    # half a step inside the grid, plus the clipped overshoot at the top
    bound = sf / 2 + np.maximum(a - qm * sf, 0) + 1e-12
    assert np.all(np.abs(x - xh) <= bound)


@pytest.mark.parametrize("b", [2, 3, 4, 7])
def test_grid_values_round_trip_exactly(b):
    rng = np.random.default_rng(b)
    qm = (1 << (b - 1)) - 1
    k = rng.integers(-qm, qm + 1, size=(16, 128))
    k[:, 5] = qm                                        # top level reached
    x = (k * 2.0 ** -3).astype(F32)
    u, s = quant.rtn_quant(x, b)
    assert np.all(s.astype(np.float64) == 2.0 ** -3)
    assert np.array_equal(u - (1 << (b - 1)), k)
    assert np.array_equal(quant.rtn_dequant(u, s, b), x.astype(np.float64))


@pytest.mark.parametrize("b", [2, 4])
def test_sign_and_power_of_two_symmetry(b):
    x = _tokens(30 + b)
    u, s = quant.rtn_quant(x, b)
    un, sn = quant.rtn_quant(-x, b)
    off = 1 << (b - 1)
    assert np.array_equal(s, sn)
    assert np.array_equal(un - off, -(u - off))       # rint is symmetric
    u4, s4 = quant.rtn_quant(x * F32(4.0), b)
    assert np.array_equal(u4, u)
    assert np.array_equal(s4.astype(np.float64), 4.0 * s.astype(np.float64))


def test_zero_token_and_one_bit_rejected():
    x = _tokens(40, T=4)
    x[2] = 0.0
    u, s = quant.rtn_quant(x, 3)
    assert s[2] == 0 and np.all(u[2] == 4)
    assert np.all(quant.rtn_dequant(u, s, 3)[2] == 0.0)
    with pytest.raises(ValueError):
        quant.rtn_quant(x, 1)


def test_quarot_is_rtn_of_the_rotated_vector():
    # QuaRot = Hadamard rotation followed by the same per-token step.
    x = _tokens(50)
    for b in (3, 4):
        uq, sq = quant.quarot_quant(x, b)
        ur, sr = quant.rtn_quant(quant.quarot_rotate(x), b)
        assert np.array_equal(uq, ur) and np.array_equal(sq, sr)


def test_cache_unit_and_sweep():
    rng = np.random.default_rng(7)
    T, R = 160, 32
    k = rng.standard_normal((T, 128)).astype(np.float16).astype(F32)
    v = rng.standard_normal((T, 128)).astype(np.float16).astype(F32)
    u = cache.Unit(cache.RTN, k, v, 3, 5, R)
    assert u.nq == 128
    kh = u.keys()
    assert kh.shape == (T, 128)
    assert np.array_equal(kh[u.nq:], k[u.nq:].astype(np.float64))
    # the quantized prefix satisfies the RTN error bound token by token
    _, s = quant.rtn_quant(k[:u.nq], 3)
    amax = np.max(np.abs(k[:u.nq].astype(np.float64)), axis=1, keepdims=True)
    assert np.all(np.abs(kh[:u.nq] - k[:u.nq])
                  <= s.astype(np.float64)[:, None] / 2 + 2.0 ** -11 * amax)
    # sweep: MSE falls with every extra bit, by about 4x at high widths
    D = calib.sweep(calib.RTN, k[None], [2, 3, 4, 5, 6, 7, 8], False)[0]
    assert np.all(np.diff(D) < 0)
    ratio = D[3:-1] / D[4:]
    assert np.all((ratio > 3.0) & (ratio < 5.0))
