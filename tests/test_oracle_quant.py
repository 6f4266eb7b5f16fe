"""Pins of the quantizer, format and cache oracles."""
import math

import numpy as np
import pytest

import workloads
from oracle import cache, fmt, quant

F32 = np.float32


def _f32(x):
    return np.asarray(x, dtype=F32)


# ---------------------------------------------------------------- format
@pytest.mark.parametrize("b", range(1, 9))
def test_pack_unpack_identity(b):
    rng = np.random.default_rng(b)
    c = rng.integers(0, 1 << b, size=(7, 3, 32))
    w = fmt.pack_chunks(c, b)
    assert w.shape == (7, 3, b) and w.dtype == np.uint32
    assert np.array_equal(fmt.unpack_chunks(w, b), c)


def test_pack_hand_examples():
    # Worked by hand from the format definition.
    c = np.arange(32) % 16                                  # b = 4
    assert [int(x) for x in fmt.pack_chunks(c, 4)] == [
        0x32103210, 0x76547654, 0xBA98BA98, 0xFEDCFEDC]
    c = np.zeros(32, dtype=int)                             # b = 1
    c[0], c[15], c[16], c[31] = 1, 1, 1, 1
    assert [int(x) for x in fmt.pack_chunks(c, 1)] == [0x80018001]
    c = np.zeros(32, dtype=int)                             # b = 3: one field
    c[0], c[16], c[9] = 7, 5, 2
    w = [int(x) for x in fmt.pack_chunks(c, 3)]
    # code 0 at stream bit 0, code 16 at bit 12 (quarter 0), code 9 =
    # quarter 2 slot 1 at bit 48 + 3 = word 1 bit 19
    assert w == [0x00005007, 0x00100000, 0x00000000]
    c = np.zeros(32, dtype=int)
    c[6], c[25], c[31] = 7, 5, 6
    w = [int(x) for x in fmt.pack_chunks(c, 3)]
    # code 6 = quarter 1 slot 2 at bits 30..32 (crosses into word 1),
    # code 25 = quarter 2 upper slot 1 at bits 63..65 (crosses into word 2),
    # code 31 = quarter 3 upper slot 3 at bits 93..95
    assert w == [0xC0000000, 0x80000001, 0xC0000002]


def test_pack3_pairs_after_spreading():
    # The property the layout is built for: quarter q's 24 bits, the upper
    # 12 moved up by 4, hold codes (4q + i, 16 + 4q + i) at bits (3i, 16 + 3i).
    rng = np.random.default_rng(3)
    c = rng.integers(0, 8, size=32)
    w = [int(x) for x in fmt.pack_chunks(c, 3)]
    stream = w[0] | (w[1] << 32) | (w[2] << 64)
    for q in range(4):
        x = (stream >> (24 * q)) & 0xFFFFFF
        z = (x & 0xFFF) | ((x >> 12) << 16)
        for i in range(4):
            assert (z >> (3 * i)) & 7 == c[4 * q + i]
            assert (z >> (16 + 3 * i)) & 7 == c[16 + 4 * q + i]


def test_plane_widths():
    assert [sum(fmt.planes(b)) for b in range(1, 9)] == list(range(1, 9))
    assert fmt.planes(7) == [4, 2, 1] and fmt.planes(6) == [4, 2]
    assert fmt.planes(3) == [3]


def test_pair_order():
    x = np.arange(32)
    p = fmt.to_pair_order(x)
    assert list(p[:6]) == [0, 16, 1, 17, 2, 18]
    assert np.array_equal(fmt.from_pair_order(p), x)


def test_f16_saturating_rounding():
    v = fmt.f16_sat(_f32([70000.0, -1e30, 1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11]))
    assert list(v.astype(np.float64)) == [65504.0, -65504.0, 1.0,
                                          1.0 + 2 * 2.0 ** -10]


# ------------------------------------------------------------------ KIVI
@pytest.mark.parametrize("b", range(1, 9))
def test_kivi_codes_in_range_and_min_exact(b):
    x = workloads.u16_to_f32(workloads.calib_cpu(2, 64, workloads.F16)[0],
                             workloads.F16)
    for fn in (quant.kivi_quant_keys, quant.kivi_quant_values):
        u, s, z = fn(x, b)
        assert u.min() >= 0 and u.max() <= (1 << b) - 1
    # fp16 inputs: z is the exact group minimum, which encodes to 0
    u, s, z = quant.kivi_quant_values(x, b)
    g = x.reshape(-1, 4, 32)
    amin = np.argmin(g, axis=-1)
    assert np.all(np.take_along_axis(u.reshape(-1, 4, 32), amin[..., None],
                                     -1) == 0)
    assert np.array_equal(z.astype(F32), g.min(axis=-1))


@pytest.mark.parametrize("b", [1, 2, 3, 4, 8])
def test_kivi_lossless_grid(b):
    # Inputs on the grid z + k s with s a power of two and k spanning
    # 0 .. 2^b - 1 round-trip exactly.
    rng = np.random.default_rng(b)
    T = 64
    k = rng.integers(0, 1 << b, size=(T // 4, 4, 32))
    k[:, :, 0] = 0
    k[:, :, 1] = (1 << b) - 1
    s = 2.0 ** rng.integers(-6, 2, size=(T // 4, 4, 1))
    z = rng.integers(-8, 8, size=(T // 4, 4, 1)) * 0.5
    x = _f32(z + k * s).reshape(T // 4, 128)
    u, ss, zz = quant.kivi_quant_values(x, b)
    assert np.array_equal(u.reshape(k.shape), k)
    xh = quant.kivi_dequant_values(u, ss, zz)
    assert np.array_equal(xh, x.astype(np.float64))


@pytest.mark.parametrize("b", [1, 2, 3, 4, 6, 8])
def test_kivi_error_bound(b):
    # |x - x_hat| <= s/2 + (2^b - 1)|s_exact - s| + |z - min|:
    # rounding to the grid plus the clamp of the top element when s was
    # rounded down, plus the rounding of the zero point.
    x = workloads.u16_to_f32(workloads.calib_cpu(2, 256, workloads.BF16)[0],
                             workloads.BF16)
    u, s, z = quant.kivi_quant_keys(x, b)
    xh = quant.kivi_dequant_keys(u, s, z)
    g = x.reshape(-1, 32, 128)
    mn, mx = g.min(axis=1).astype(np.float64), g.max(axis=1).astype(np.float64)
    s64, z64 = s.astype(np.float64), z.astype(np.float64)
    s_exact = (mx - z64) / ((1 << b) - 1)
    bound = s64 / 2 + ((1 << b) - 1) * np.abs(s_exact - s64) + np.abs(z64 - mn)
    err = np.abs(x.astype(np.float64) - xh).reshape(-1, 32, 128)
    assert np.all(err <= bound[:, None, :] * (1 + 1e-6) + 1e-30)


def test_kivi_constant_group():
    x = np.full((32, 128), 1.5, dtype=F32)
    u, s, z = quant.kivi_quant_keys(x, 3)
    assert np.all(u == 0) and np.all(s.astype(F32) == 0)
    assert np.all(quant.kivi_dequant_keys(u, s, z) == 1.5)


def test_kivi_high_bit_mse_is_uniform_noise():
    # At b = 8 the rounding error is ~uniform on [-s/2, s/2] (MSE s^2 / 12)
    # except for the group minimum and maximum, which are (nearly) exact:
    # MSE ~ (30 / 32) s^2 / 12.
    x = workloads.u16_to_f32(workloads.calib_cpu(2, 1024, workloads.F16)[1],
                             workloads.F16)
    u, s, z = quant.kivi_quant_values(x, 8)
    xh = quant.kivi_dequant_values(u, s, z)
    mse = np.mean((x - xh) ** 2)
    want = np.mean(s.astype(np.float64) ** 2) / 12 * 30 / 32
    assert abs(mse / want - 1) < 0.02


# ---------------------------------------------------------------- QuaRot
def test_hadamard_orthogonality_and_fwht():
    H = quant.hadamard()
    assert np.array_equal(H @ H.T, 128 * np.eye(128))
    e0 = np.zeros(128, dtype=F32)
    e0[0] = 1
    assert np.array_equal(quant.fwht_f32(e0), np.ones(128, dtype=F32))
    rng = np.random.default_rng(0)
    xi = rng.integers(-50, 50, size=(16, 128)).astype(F32)
    # integers: every fp32 step is exact, so the transform equals H x and
    # applying it twice gives 128 x
    assert np.array_equal(quant.fwht_f32(xi).astype(np.float64),
                          xi.astype(np.float64) @ H.T)
    assert np.array_equal(quant.fwht_f32(quant.fwht_f32(xi)), 128 * xi)


def test_rotation_preserves_norm():
    x = workloads.u16_to_f32(workloads.calib_cpu(2, 64, workloads.BF16)[0],
                             workloads.BF16)
    y = quant.quarot_rotate(x)
    np.testing.assert_allclose(np.linalg.norm(y, axis=1),
                               np.linalg.norm(x, axis=1), rtol=1e-5)
    assert quant.INV_SQRT_D_F32.view(np.uint32) == 0x3DB504F3


@pytest.mark.parametrize("b", [2, 3, 4, 5, 6, 8])
def test_quarot_codes(b):
    x = workloads.u16_to_f32(workloads.calib_cpu(2, 128, workloads.BF16)[0],
                             workloads.BF16)
    u, s = quant.quarot_quant(x, b)
    qm = (1 << (b - 1)) - 1
    assert u.min() >= 1 and u.max() <= 2 * qm + 1
    y = quant.quarot_rotate(x)
    # the largest-magnitude coordinate takes the extreme level
    i = np.argmax(np.abs(y), axis=1)
    q = np.take_along_axis(u, i[:, None], 1)[:, 0] - (1 << (b - 1))
    assert np.all(np.abs(q) == qm)
    # sign symmetry: rint is odd, so codes of -x mirror those of x
    u2, s2 = quant.quarot_quant(-x, b)
    assert np.array_equal(s2, s) and np.array_equal(u2, (1 << b) - u)
    # rotated-domain error within half a step plus the clamp term
    yh = (u - (1 << (b - 1))) * s.astype(np.float64)[:, None]
    a = np.max(np.abs(y), axis=1).astype(np.float64)
    s64 = s.astype(np.float64)
    bound = s64 / 2 + qm * np.abs(a / qm - s64)
    assert np.all(np.abs(y - yh) <= bound[:, None] * (1 + 1e-6))
    # and the original-domain dequantization is the inverse rotation
    xh = quant.quarot_dequant(u, s, b)
    np.testing.assert_allclose(np.linalg.norm(x - xh, axis=1),
                               np.linalg.norm(y - yh, axis=1), rtol=1e-4,
                               atol=1e-6)


def test_quarot_rejects_one_bit():
    with pytest.raises(ValueError):
        quant.quarot_quant(np.ones((1, 128), dtype=F32), 1)


# ------------------------------------------------------------------ cache
def test_residual_rule():
    assert cache.n_quantized(1024, 32) == 992
    assert cache.n_quantized(131072, 128) == 130944
    assert cache.n_quantized(131072 + 31, 128) == 130944
    assert cache.n_quantized(131072 + 32, 128) == 130976
    assert cache.n_quantized(10, 32) == 0
    assert cache.n_quantized(32768, 0) == 32768


def test_unit_layout_roundtrip_and_bytes():
    wl = workloads.SMALL
    k16, v16 = workloads.kv_cpu(wl, 0, 0, 256)
    k = workloads.u16_to_f32(k16[1], wl.dtype)
    v = workloads.u16_to_f32(v16[1], wl.dtype)
    u = cache.Unit(cache.KIVI, k, v, 3, 2, 32)
    assert u.nq == 224
    assert u.k_words.shape == (224, 4, 3) and u.v_words.shape == (7, 128, 2)
    assert np.array_equal(cache.unpack_keys(u.k_words, 3), u.k_codes)
    assert np.array_equal(cache.unpack_values(u.v_words, 2), u.v_codes)
    # code bytes are exactly b bits per quantized element
    assert u.k_words.nbytes == 224 * 128 * 3 // 8
    assert u.v_words.nbytes == 224 * 128 * 2 // 8
    assert u.k_meta.shape == (7, 4, 2, 32) and u.v_meta.shape == (7, 4, 2, 32)
    assert u.keys().shape == (256, 128)
    np.testing.assert_array_equal(u.keys()[224:], k[224:])


def test_memory_footprint_accounting():
    # Appendix "Memory Footprint": Qwen3-8B KV at 4096 tokens is 576 MB in
    # FP16 and 144 MB at 4 bits (code bits only), 126 MB at 3.5 bits.
    L, H, T, d = 36, 8, 4096, 128
    fp16 = 2 * L * H * T * d * 2
    assert round(fp16 / 2 ** 20) == 576
    bits = 4
    codes = 2 * L * H * (T // 32) * 128 * bits * 4
    assert codes * 4 == fp16 and round(codes / 2 ** 20) == 144
    assert round(fp16 * 3.5 / 16 / 2 ** 20) == 126
