"""GPU parity of the TurboQuant-style path (through the C-ABI) against the
oracle.  Norms, the residual window and every code away from a threshold
are exact; the rotation runs on the matrix cores in fp32, so a coordinate
whose t lies within that arithmetic's error bound of a threshold may take
the adjacent code (bound: 128 * 2^-24 * sum_c |R||x| * sqrt(128) / n, twice,
plus 2^-22 |t| for the scaling)."""
import math

import numpy as np
import pytest

import paper_2605_06675_amd as rq
import workloads
from oracle import cache as ocache
from oracle import quant as oquant
from tests import gpu_helpers as gh

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return torch


def _rotations(L, H, seed=42):
    r16 = np.stack([np.stack([workloads.turbo_rotation(seed, l, h)
                              for h in range(H)]) for l in range(L)])
    return r16, workloads.u16_to_f32(r16, workloads.BF16).astype(np.float64)


def _build(dtype, H, T, R, bits, batch, chunks=None, seed=42, G=2):
    torch = _torch()
    r16, rf = _rotations(1, H, seed)
    wl = workloads.Workload("t", workloads.TURBO, dtype, 1, batch, H, G * H,
                            T, R, (1,), 2.0, 0.5, (1.0, 1.0))
    cap = ((T + 31) // 32) * 32
    kvc = rq.KVCache(rq.RQ_TURBO, dtype, 1, batch, H, G * H, cap, R, bits,
                     rotation=gh.dev(r16, workloads.BF16))
    ks, vs = zip(*[workloads.kv_cpu(wl, 0, b, T, seed=seed) for b in range(batch)])
    K, V = gh.dev(np.stack(ks), dtype), gh.dev(np.stack(vs), dtype)
    t0 = 0
    for n in chunks or [T]:
        kvc.append(0, K[:, :, t0:t0 + n].contiguous(), V[:, :, t0:t0 + n].contiguous())
        t0 += n
    torch.cuda.synchronize()
    return kvc, ks, vs, rf[0]


def _eps(x, R, n16, t):
    """Per-element bound on |t_gpu - t| (see the module docstring)."""
    x = np.asarray(x, np.float64)
    s = np.abs(x) @ np.abs(R).T
    n = np.asarray(n16, np.float64)[:, None]
    scale = np.where(n > 0, math.sqrt(128.0) / np.where(n > 0, n, 1.0), 0.0)
    return 2.0 * 128 * 2.0 ** -24 * s * scale + 2.0 ** -22 * np.abs(t)


def _compare_codes(got, want, t, b, eps, what):
    diff = got.astype(np.int64) - want
    bad = diff != 0
    if bad.any():
        assert np.all(np.abs(diff[bad]) == 1), f"{what}: non-adjacent code"
        near = oquant.turbo_near_threshold(t[bad], b, eps[bad])
        assert near.all(), (f"{what}: {np.count_nonzero(~near)} code(s) differ "
                            f"away from a threshold")
    return int(np.count_nonzero(bad))


def _check(dtype, kvc, ks, vs, Rf, bits, R, batch, H):
    lay = gh.Layout(gh.TURBO, 1, batch, H, kvc.desc.capacity, R, bits)
    codes_u8, meta_u8, resid_u16 = gh.read_buffers(kvc)
    total = mism = 0
    units = {}
    for b in range(batch):
        for h in range(H):
            bk, bv = int(bits[0, h, 0]), int(bits[0, h, 1])
            k = workloads.u16_to_f32(ks[b][h], dtype)
            v = workloads.u16_to_f32(vs[b][h], dtype)
            u = ocache.Unit(ocache.TURBO, k, v, bk, bv, R, rotation=Rf[h])
            units[(b, h)] = u
            nq = u.nq
            for kind, want_meta in ((0, u.k_meta), (1, u.v_meta)):
                got = lay.meta(meta_u8, 0, b, h, kind, nq // 32)
                np.testing.assert_array_equal(got.view(np.uint16),
                                              np.asarray(want_meta).view(np.uint16))
            gk = ocache.unpack_keys(lay.k_words(codes_u8, 0, b, h, nq), bk)
            gv = ocache.unpack_values(lay.v_words(codes_u8, 0, b, h, nq // 32), bv)
            nk = oquant.turbo_norm(k[:nq])
            nv = oquant.turbo_norm(v[:nq])
            mism += _compare_codes(gk, u.k_codes, u.k_t, bk,
                                   _eps(k[:nq], Rf[h], nk, u.k_t), f"K b{b} h{h}")
            mism += _compare_codes(gv, u.v_codes, u.v_t, bv,
                                   _eps(v[:nq], Rf[h], nv, u.v_t), f"V b{b} h{h}")
            total += 2 * nq * 128
            for kind, src in ((0, ks[b][h]), (1, vs[b][h])):
                ring = lay.ring(resid_u16, 0, b, h, kind)
                for t in range(nq, u.T):
                    np.testing.assert_array_equal(ring[ocache.ring_slot(t, R)], src[t])
    print(f"codes {total}, adjacent near-threshold differences {mism}")
    assert mism <= max(2, total // 1000)
    return units


@pytest.mark.parametrize("dtype", [workloads.BF16, workloads.F16])
def test_turbo_quantize_narrow_widths(dtype):
    bits = np.array([[[1, 2], [2, 3], [3, 4], [4, 1]]])
    kvc, ks, vs, Rf = _build(dtype, 4, 200, 32, bits, 2)
    _check(dtype, kvc, ks, vs, Rf, bits, 32, 2, 4)


def test_turbo_quantize_wide_widths_chunked():
    bits = np.array([[[5, 6], [7, 8]]])
    kvc, ks, vs, Rf = _build(workloads.BF16, 2, 230, 40, bits, 1,
                             chunks=[70, 1, 100, 59])
    _check(workloads.BF16, kvc, ks, vs, Rf, bits, 40, 1, 2)


def test_turbo_quantize_many_blocks_per_wave():
    # 4 x 8 units of 2048 tokens: every wave of the persistent kernel loops
    bits = np.array([[[2 + h % 3, 4 - h % 3] for h in range(8)]])
    kvc, ks, vs, Rf = _build(workloads.BF16, 8, 2048, 0, bits, 4)
    _check(workloads.BF16, kvc, ks, vs, Rf, bits, 0, 4, 8)


def _attention(kvc, units, dtype, batch, H, G, seed=7, q_mult=1.0):
    torch = _torch()
    from oracle import attention as oatt
    from tests.test_gpu_parity import attention_tol
    q16 = np.random.default_rng(seed).standard_normal((batch, H * G, 128)) * q_mult
    q16 = workloads.bits16_from_f32(q16, dtype)
    out = kvc.attention(0, gh.dev(q16, dtype))
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    assert np.all(np.isfinite(out))
    worst = 0.0
    for (b, h), u in units.items():
        q = workloads.u16_to_f32(q16[b, h * G:(h + 1) * G], dtype)
        v_hat = u.values()
        want = oatt.decode_attention(q, u.keys(), v_hat)
        err = float(np.max(np.abs(out[b, h * G:(h + 1) * G] - want)))
        tol = attention_tol(v_hat)
        assert err < tol, (b, h, err, tol)
        worst = max(worst, err / tol * 1e-2)
    print(f"attention max-abs error {worst:.3e} (at unit scale)")
    return worst


@pytest.mark.parametrize("dtype", [workloads.BF16, workloads.F16])
def test_turbo_attention_every_narrow_width(dtype):
    bits = np.array([[[1, 2], [2, 3], [3, 4], [4, 1]]])
    kvc, ks, vs, Rf = _build(dtype, 4, 300, 32, bits, 2)
    units = _check(dtype, kvc, ks, vs, Rf, bits, 32, 2, 4)
    _attention(kvc, units, dtype, 2, 4, 2)


def test_turbo_attention_eight_queries_per_head_no_window():
    # the Llama-3-70B shape per kv-head: G = 8, window 0, bits {2, 3, 4}
    bits = np.array([[[2 + h % 3, 4 - h % 3] for h in range(8)]])
    kvc, ks, vs, Rf = _build(workloads.BF16, 8, 1500, 0, bits, 2, G=8)
    units = _check(workloads.BF16, kvc, ks, vs, Rf, bits, 0, 2, 8)
    _attention(kvc, units, workloads.BF16, 2, 8, 8)


@pytest.mark.parametrize("G", [3, 6])
def test_turbo_attention_group_sizes_not_power_of_two(G):
    # query heads per kv-head that leave rotated query rows unused (3 of 4,
    # 6 of 8); pair-table widths 2..4 and a centroid-table width; 1100
    # tokens so several streaming workgroups merge
    bits = np.array([[[2, 3], [4, 2], [3, 5]]])
    print(f"turbo group size {G}", flush=True)
    kvc, ks, vs, Rf = _build(workloads.BF16, 3, 1100, 32, bits, 2, G=G)
    units = _check(workloads.BF16, kvc, ks, vs, Rf, bits, 32, 2, 3)
    _attention(kvc, units, workloads.BF16, 2, 3, G)


@pytest.mark.parametrize("dtype", [workloads.BF16, workloads.F16])
def test_turbo_attention_wide_widths(dtype):
    # widths 5..8 look their centroids up in LDS; mixed with narrow ones
    bits = np.array([[[5, 6], [7, 8], [6, 3], [2, 5]]])
    kvc, ks, vs, Rf = _build(dtype, 4, 300, 32, bits, 2, G=4)
    units = _check(dtype, kvc, ks, vs, Rf, bits, 32, 2, 4)
    _attention(kvc, units, dtype, 2, 4, 4)


def test_turbo_attention_paper_bounds_3_to_6():
    """The paper's bit-width bounds at 3.5 bits (Appendix "Implementation
    Details": [3, 6] for b >= 3.5): a Llama-3-70B-shaped layer per kv-head
    (8 query heads each, no window) with bits allocated by rq_allocate_bits
    over 16 components."""
    rng = np.random.default_rng(5)
    n = 16
    w = rng.lognormal(0.0, 0.74, n)
    beta = rng.uniform(3.6, 5.3, n)
    alpha = np.full(n, 1.5)
    bits, _, _ = rq.rq_allocate_bits(w, alpha, beta, 3.5, 3, 6)
    assert bits.sum() == 56 and bits.min() >= 3 and bits.max() <= 6
    assert bits.max() >= 5
    table = bits.reshape(1, 8, 2)
    kvc, ks, vs, Rf = _build(workloads.BF16, 8, 1500, 0, table, 2, G=8)
    units = _check(workloads.BF16, kvc, ks, vs, Rf, table, 0, 2, 8)
    _attention(kvc, units, workloads.BF16, 2, 8, 8)


@pytest.mark.parametrize("dtype,bits", [(workloads.BF16, [1, 2, 3, 4]),
                                        (workloads.F16, [2, 3, 4, 5, 6])])
def test_turbo_calibration_sweep(dtype, bits):
    """8 components x 512 tokens, each with its own rotation: the error is
    measured in the original domain (x - R^T y_hat) like the oracle's."""
    torch = _torch()
    from oracle import calib as ocalib
    from oracle import fit as ofit
    x16 = workloads.calib_cpu(8, 512, dtype)
    x = workloads.u16_to_f32(x16, dtype)
    r16 = np.stack([workloads.turbo_rotation(42, 0, i) for i in range(8)])
    rf = workloads.u16_to_f32(r16, workloads.BF16).astype(np.float64)
    cb = torch.from_numpy(rq.rq_turbo_codebook().reshape(-1)).cuda()
    mse, a, b, _ = rq.rq_calibrate_distortion(
        rq.RQ_TURBO, dtype, gh.dev(x16, dtype), 0, bits,
        rotation=gh.dev(r16, workloads.BF16), codebook=cb)
    want = ocalib.sweep(ocalib.TURBO, x, bits, False, rf)
    rel = np.abs(mse / want - 1)
    print(f"turbo sweep: max rel {rel.max():.2e}")
    assert np.all(rel <= 1e-5)
    wa, wb, _ = ofit.fit_distortion(want, bits)
    np.testing.assert_allclose(b, wb, rtol=1e-4)


def test_turbo_attention_two_level_merge():
    # batch 1, two kv-heads, 4096 tokens: partials merged in groups first
    bits = np.array([[[3, 2], [4, 3]]])
    kvc, ks, vs, Rf = _build(workloads.BF16, 2, 4096, 64, bits, 1, G=8)
    units = _check(workloads.BF16, kvc, ks, vs, Rf, bits, 64, 1, 2)
    _attention(kvc, units, workloads.BF16, 1, 2, 8)
