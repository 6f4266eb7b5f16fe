"""GPU parity: the HIP path (through the C-ABI) against the oracle on the
same seeded inputs.  Packed codes, metadata and the residual window must be
bit-exact; attention outputs within 1e-2 max-abs; sweep MSE within a
relative 2^(b-21) (fp32 error of one element, see the design notes)."""
import math

import numpy as np
import pytest

import paper_2605_06675_amd as rq
import workloads
from oracle import attention as oatt
from oracle import cache as ocache
from oracle import calib as ocalib
from oracle import fit as ofit
from tests import gpu_helpers as gh

pytestmark = pytest.mark.gpu

ATOL = 1e-2


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return torch


def _unit_inputs(wl, l, b, T, seed=42):
    k16, v16 = workloads.kv_cpu(wl, l, b, T, seed=seed)
    return k16, v16


def _build(family, dtype, H, G, T, R, bits, batch=1, seed=42, cap=None,
           chunks=None):
    """Fill a one-layer cache with T tokens (in the given append chunks)
    and return (cache object, per-batch uint16 inputs)."""
    torch = _torch()
    wl = workloads.Workload("t", family, dtype, 1, batch, H, H * G, T, R,
                            (1,), 2.0, 0.5, (1.0, 1.0))
    cap = cap or ((T + 31) // 32) * 32
    kvc = rq.KVCache(family, dtype, 1, batch, H, H * G, cap, R, bits)
    ks, vs = [], []
    for b in range(batch):
        k16, v16 = _unit_inputs(wl, 0, b, T, seed)
        ks.append(k16)
        vs.append(v16)
    K = gh.dev(np.stack(ks), dtype)      # [B][H][T][128]
    V = gh.dev(np.stack(vs), dtype)
    chunks = chunks or [T]
    t0 = 0
    for n in chunks:
        kvc.append(0, K[:, :, t0:t0 + n].contiguous(),
                   V[:, :, t0:t0 + n].contiguous())
        t0 += n
    assert t0 == T
    torch.cuda.synchronize()
    return kvc, ks, vs, wl


def _check_cache(family, dtype, kvc, ks, vs, bits, R, batch, H, T):
    lay = gh.Layout(family, 1, batch, H, kvc.desc.capacity, R, bits)
    bufs = gh.read_buffers(kvc)
    units = {}
    for b in range(batch):
        for h in range(H):
            k = workloads.u16_to_f32(ks[b][h], dtype)
            v = workloads.u16_to_f32(vs[b][h], dtype)
            u = ocache.Unit(family, k, v, int(bits[0, h, 0]),
                            int(bits[0, h, 1]), R)
            gh.compare_unit(lay, bufs, 0, b, h, u, ks[b][h], vs[b][h])
            units[(b, h)] = u
    return units


def attention_tol(v_hat):
    """Attention tolerance of one unit: 1e-2 max-abs for values of the
    workloads' unit scale, growing in proportion to the values beyond it
    (fp16 operands carry 11 significant bits whatever the magnitude)."""
    return ATOL * max(1.0, float(np.max(np.abs(v_hat))) / 8.0)


def _check_attention(kvc, units, dtype, batch, H, G, seed=7, q_mult=1.0):
    torch = _torch()
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
        err = np.max(np.abs(out[b, h * G:(h + 1) * G] - want))
        assert err < attention_tol(v_hat), (b, h, err, attention_tol(v_hat))
        worst = max(worst, err / attention_tol(v_hat) * ATOL)
    print(f"attention max-abs error {worst:.3e} (at unit scale)")
    return worst


# --------------------------------------------------------------------- KIVI
def test_small_workload_kivi_fp16():
    """Single layer, batch 1, 8 kv-heads, 32 q-heads, 1024 tokens, fp16,
    KIVI g32, 32-token window, bits [4,2,2,3,2,2,3,2] for K and V."""
    wl = workloads.SMALL
    hb = np.array(wl.fixed_bits)
    bits = np.stack([hb, hb], axis=-1)[None]
    kvc, ks, vs, _ = _build(workloads.KIVI, workloads.F16, 8, 4, 1024, 32,
                            bits)
    units = _check_cache(workloads.KIVI, workloads.F16, kvc, ks, vs, bits, 32,
                         1, 8, 1024)
    assert units[(0, 0)].nq == 992
    _check_attention(kvc, units, workloads.F16, 1, 8, 4)


@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
def test_kivi_every_bit_width_ragged(dtype):
    # head h: K at h+1 bits, V at 8-h bits; 200 tokens, window 32 ->
    # 160 quantized + 40 in the window
    bits = np.array([[[h + 1, 8 - h] for h in range(8)]])
    kvc, ks, vs, _ = _build(workloads.KIVI, dtype, 8, 2, 200, 32, bits,
                            batch=2, cap=256)
    units = _check_cache(workloads.KIVI, dtype, kvc, ks, vs, bits, 32, 2, 8,
                         200)
    _check_attention(kvc, units, dtype, 2, 8, 2)


@pytest.mark.parametrize("wide", [False, True])
def test_kivi_many_blocks_per_wave(wide):
    # Enough blocks that every wave of the persistent quantize kernel loops
    # several times (8192 blocks); layers with widths up to 4 and up to 8
    # take different kernel instances.
    H, batch, T = 8, 4, 4128
    if wide:
        bits = np.array([[[h + 1, 8 - h] for h in range(H)]])
    else:
        bits = np.array([[[1 + h % 4, 4 - h % 4] for h in range(H)]])
    kvc, ks, vs, _ = _build(workloads.KIVI, workloads.BF16, H, 1, T, 32, bits,
                            batch=batch)
    _check_cache(workloads.KIVI, workloads.BF16, kvc, ks, vs, bits, 32, batch,
                 H, T)


def test_kivi_chunked_prefill_equals_one_shot():
    bits = np.array([[[2, 3], [1, 4], [4, 2], [3, 1]]])
    kvc, ks, vs, _ = _build(workloads.KIVI, workloads.BF16, 4, 4, 301, 40,
                            bits, batch=1, cap=320, chunks=[45, 1, 70, 33, 152])
    units = _check_cache(workloads.KIVI, workloads.BF16, kvc, ks, vs, bits, 40,
                         1, 4, 301)
    _check_attention(kvc, units, workloads.BF16, 1, 4, 4)


def test_kivi_decode_steps_with_flushes():
    """Prefill 96 tokens then append one token at a time; attention after
    every step covers the blocks flushed out of the 32-token window."""
    torch = _torch()
    H, G, R, T0, steps = 2, 8, 32, 96, 70
    bits = np.array([[[3, 2], [2, 4]]])
    T = T0 + steps
    wl = workloads.Workload("t", workloads.KIVI, workloads.BF16, 1, 1, H,
                            H * G, T, R, (1,), 2.0, 0.5, (1.0, 1.0))
    k16, v16 = workloads.kv_cpu(wl, 0, 0, T)
    K, V = gh.dev(k16[None], workloads.BF16), gh.dev(v16[None], workloads.BF16)
    kvc = rq.KVCache(workloads.KIVI, workloads.BF16, 1, 1, H, H * G, 192, R,
                     bits)
    kvc.append(0, K[:, :, :T0].contiguous(), V[:, :, :T0].contiguous())
    q16 = workloads.bits16_from_f32(
        np.random.default_rng(3).standard_normal((1, H * G, 128)),
        workloads.BF16)
    qd = gh.dev(q16, workloads.BF16)
    worst = 0.0
    for s in range(steps):
        t = T0 + s
        kvc.append(0, K[:, :, t:t + 1].contiguous(), V[:, :, t:t + 1].contiguous())
        if s % 7 == 0 or s == steps - 1:
            out = kvc.attention(0, qd).cpu().numpy()
            for h in range(H):
                u = ocache.Unit(workloads.KIVI,
                                workloads.u16_to_f32(k16[h, :t + 1], workloads.BF16),
                                workloads.u16_to_f32(v16[h, :t + 1], workloads.BF16),
                                int(bits[0, h, 0]), int(bits[0, h, 1]), R)
                q = workloads.u16_to_f32(q16[0, h * G:(h + 1) * G], workloads.BF16)
                want = oatt.decode_attention(q, u.keys(), u.values())
                worst = max(worst, np.max(np.abs(out[0, h * G:(h + 1) * G] - want)))
    torch.cuda.synchronize()
    print(f"decode-step attention max-abs error {worst:.3e}")
    assert worst < ATOL
    _check_cache(workloads.KIVI, workloads.BF16, kvc, [k16], [v16], bits, R,
                 1, H, T)


@pytest.mark.parametrize("G", [4, 8])
def test_kivi_two_level_merge_long_context(G):
    """Two kv-heads, batch 1, 8000+ tokens: more than 16 workgroups per
    unit, so partials are merged in groups first.  Attention after the
    prefill and after appends that change the number of workgroups (the
    counters must be ready for the next call every time)."""
    torch = _torch()
    H, R, T0 = 2, 128, 8000
    bits = np.array([[[2, 1], [3, 4]]])
    T = T0 + 300
    wl = workloads.Workload("t", workloads.KIVI, workloads.BF16, 1, 1, H,
                            H * G, T, R, (1,), 2.0, 0.5, (1.0, 1.0))
    k16, v16 = workloads.kv_cpu(wl, 0, 0, T)
    K, V = gh.dev(k16[None], workloads.BF16), gh.dev(v16[None], workloads.BF16)
    kvc = rq.KVCache(workloads.KIVI, workloads.BF16, 1, 1, H, H * G, 8320, R, bits)
    q16 = workloads.bits16_from_f32(
        np.random.default_rng(5).standard_normal((1, H * G, 128)), workloads.BF16)
    qd = gh.dev(q16, workloads.BF16)
    worst, t = 0.0, 0
    for n in (T0, 1, 150, 149):
        kvc.append(0, K[:, :, t:t + n].contiguous(), V[:, :, t:t + n].contiguous())
        t += n
        out = kvc.attention(0, qd).cpu().numpy()
        for h in range(H):
            u = ocache.Unit(workloads.KIVI,
                            workloads.u16_to_f32(k16[h, :t], workloads.BF16),
                            workloads.u16_to_f32(v16[h, :t], workloads.BF16),
                            int(bits[0, h, 0]), int(bits[0, h, 1]), R)
            q = workloads.u16_to_f32(q16[0, h * G:(h + 1) * G], workloads.BF16)
            want = oatt.decode_attention(q, u.keys(), u.values())
            worst = max(worst, np.max(np.abs(out[0, h * G:(h + 1) * G] - want)))
    torch.cuda.synchronize()
    print(f"long-context attention max-abs error {worst:.3e}")
    assert worst < ATOL


@pytest.mark.parametrize("family,G", [(workloads.KIVI, 1), (workloads.KIVI, 3),
                                      (workloads.KIVI, 6), (workloads.QUAROT, 3),
                                      (workloads.RTN, 6)])
def test_group_sizes_not_power_of_two(family, G):
    """Query heads per kv-head that leave replicas of the query rows unused
    (3 of 4, 6 of 8) or a single row; 1100 tokens so several streaming
    workgroups merge.  KIVI's value side takes one (G <= 4) or two (G = 6)
    A operands."""
    lo = 1 if family == workloads.KIVI else 2
    bits = np.array([[[lo, 3], [4, lo], [3, 4]]])
    print(f"group size {G} family {family}", flush=True)
    kvc, ks, vs, _ = _build(family, workloads.BF16, 3, G, 1100, 32, bits,
                            batch=2)
    units = _check_cache(family, workloads.BF16, kvc, ks, vs, bits, 32, 2, 3,
                         1100)
    _check_attention(kvc, units, workloads.BF16, 2, 3, G)


@pytest.mark.parametrize("fill", ["foreign_tags", "random_bytes"])
def test_stale_workspace_counters(fill):
    """A workspace whose counters hold counts of other calls (foreign tags,
    arbitrary counts: what a call that did not finish leaves) or random
    bytes: the call replaces the stale counts and matches the oracle, and
    the call after it (on counters this call readied) does too.  4100
    tokens over 2 x 4 units: two-level merges with claims in each group."""
    torch = _torch()
    H, G, T = 4, 4, 4100
    bits = np.array([[[2, 3], [1, 4], [3, 2], [4, 1]]])
    kvc, ks, vs, _ = _build(workloads.KIVI, workloads.BF16, H, G, T, 32, bits,
                            batch=2)
    units = _check_cache(workloads.KIVI, workloads.BF16, kvc, ks, vs, bits, 32,
                         2, H, T)
    ws = kvc.workspace(T)
    rng = np.random.default_rng(17)
    n8 = ws.numel() // 8
    if fill == "foreign_tags":
        tag = rng.integers(0x40000000, 0x7fffffff, size=n8, dtype=np.int64)
        cnt = rng.integers(0, 1000, size=n8, dtype=np.int64)
        stale = torch.from_numpy((tag << 32) | cnt).to(ws.device)
        ws[:n8 * 8].view(torch.int64).copy_(stale)
    else:
        raw = rng.integers(0, 256, size=ws.numel(), dtype=np.uint8)
        ws.copy_(torch.from_numpy(raw).to(ws.device))
    torch.cuda.synchronize()
    print(f"stale workspace ({fill})", flush=True)
    for call in range(2):
        _check_attention(kvc, units, workloads.BF16, 2, H, G, seed=11 + call)


def test_short_context_window_only():
    # fewer tokens than the window: nothing quantized, attention is exact
    bits = np.array([[[2, 2], [3, 3]]])
    for T in (1, 5, 31):
        kvc, ks, vs, _ = _build(workloads.KIVI, workloads.F16, 2, 4, T, 32,
                                bits, cap=64)
        units = _check_cache(workloads.KIVI, workloads.F16, kvc, ks, vs, bits,
                             32, 1, 2, T)
        assert units[(0, 0)].nq == 0
        _check_attention(kvc, units, workloads.F16, 1, 2, 4)


@pytest.mark.parametrize("T", [100, 200, 700])
def test_window_chunks_outnumber_workgroups(T):
    # a 160-token window is 5 or 6 chunks of 32 tokens, more than the few
    # streaming workgroups of these short caches, so a workgroup takes
    # several chunks before its blocks (T=100: nothing quantized, one
    # workgroup takes every chunk; T=700: 5 workgroups, 6 chunks)
    bits = np.array([[[2, 3], [4, 1]]])
    kvc, ks, vs, _ = _build(workloads.KIVI, workloads.F16, 2, 4, T, 160,
                            bits, batch=2, cap=768)
    units = _check_cache(workloads.KIVI, workloads.F16, kvc, ks, vs, bits,
                         160, 2, 2, T)
    _check_attention(kvc, units, workloads.F16, 2, 2, 4)


def test_no_window():
    bits = np.array([[[1, 2], [4, 3]]])
    kvc, ks, vs, _ = _build(workloads.KIVI, workloads.BF16, 2, 16, 256, 0,
                            bits)
    units = _check_cache(workloads.KIVI, workloads.BF16, kvc, ks, vs, bits, 0,
                         1, 2, 256)
    assert units[(0, 1)].nq == 256
    _check_attention(kvc, units, workloads.BF16, 1, 2, 16)


# ------------------------------------------------------------------- QuaRot
@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
def test_quarot_every_bit_width(dtype):
    bits = np.array([[[h + 2, 8 - h] for h in range(7)]])
    kvc, ks, vs, _ = _build(workloads.QUAROT, dtype, 7, 4, 160, 0, bits,
                            batch=2)
    units = _check_cache(workloads.QUAROT, dtype, kvc, ks, vs, bits, 0, 2, 7,
                         160)
    _check_attention(kvc, units, dtype, 2, 7, 4)


def test_quarot_with_window_and_ragged_tail():
    bits = np.array([[[4, 5], [6, 3]]])
    kvc, ks, vs, _ = _build(workloads.QUAROT, workloads.BF16, 2, 8, 333, 16,
                            bits, cap=352, chunks=[100, 200, 1, 32])
    units = _check_cache(workloads.QUAROT, workloads.BF16, kvc, ks, vs, bits,
                         16, 1, 2, 333)
    _check_attention(kvc, units, workloads.BF16, 1, 2, 8)


# -------------------------------------------------------------- calibration
@pytest.mark.parametrize("family,bits", [(workloads.KIVI, [1, 2, 3, 4]),
                                         (workloads.KIVI, [5, 6, 7, 8]),
                                         (workloads.QUAROT, [2, 3, 4, 5, 6])])
def test_calibration_sweep(family, bits):
    """8 key + 8 value components x 512 tokens (the single-layer workload's
    calibration case)."""
    _torch()
    dtype = workloads.F16
    x16 = workloads.calib_cpu(16, 512, dtype)
    x = workloads.u16_to_f32(x16, dtype)
    for is_value, sl in ((0, slice(0, 8)), (1, slice(8, 16))):
        mse, a, b, r2 = rq.rq_calibrate_distortion(
            family, dtype, gh.dev(np.ascontiguousarray(x16[sl]), dtype),
            is_value, bits)
        want = ocalib.sweep(family, x[sl], bits, bool(is_value))
        tol = np.array([2.0 ** (bb - 21) for bb in bits])
        rel = np.abs(mse / want - 1)
        print(f"sweep family {family} value {is_value}: max rel {rel.max():.2e}")
        assert np.all(rel <= tol[None, :])
        wa, wb, wr = ofit.fit_distortion(want, bits)
        np.testing.assert_allclose(a, wa, rtol=1e-4)
        np.testing.assert_allclose(b, wb, rtol=1e-4)


# --------------------------------------------- full-size layer, sampled units
def test_llama3_8b_layer_sampled():
    """One full layer of the Llama-3-8B shaped workload (batch 16, 8192
    tokens, bf16, KIVI g32, window 32, bits from the allocator at 2.5
    average), checked on sampled units, one of every width pair of the layer
    among them."""
    torch = _torch()
    wl = workloads.LLAMA3_8B
    w, a, be = workloads.allocation_inputs(wl)
    alloc_bits, _, _ = rq.rq_allocate_bits(w, a, be, wl.avg_bits, 1, 4)
    bits = alloc_bits.reshape(wl.n_layers, wl.n_kv_heads, 2)[:1]
    layer = 0
    K, V = workloads.kv_device(wl, layer)
    kvc = rq.KVCache(wl.family, wl.dtype, 1, wl.batch, wl.n_kv_heads,
                     wl.n_q_heads, wl.context, wl.residual, bits)
    kvc.append(0, K, V)
    qd = workloads.q_device(wl, layer)
    out = kvc.attention(0, qd)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    q16 = gh.host_bits(qd)
    lay = gh.Layout(wl.family, 1, wl.batch, wl.n_kv_heads, wl.context,
                    wl.residual, bits)
    bufs = gh.read_buffers(kvc)
    G = wl.group
    worst = 0.0
    # three fixed units, plus one unit of every (K, V) width pair of the layer
    first_of_pair = {}
    for h in range(wl.n_kv_heads):
        first_of_pair.setdefault(tuple(int(x) for x in bits[0, h]), h)
    units = {(0, 0), (7, 3), (15, 7)}
    units |= {((5 * h) % wl.batch, h) for h in first_of_pair.values()}
    for (b, h) in sorted(units):
        k16 = gh.host_bits(K[b, h])
        v16 = gh.host_bits(V[b, h])
        u = ocache.Unit(wl.family, workloads.u16_to_f32(k16, wl.dtype),
                        workloads.u16_to_f32(v16, wl.dtype),
                        int(bits[0, h, 0]), int(bits[0, h, 1]), wl.residual)
        gh.compare_unit(lay, bufs, 0, b, h, u, k16, v16)
        q = workloads.u16_to_f32(q16[b, h * G:(h + 1) * G], wl.dtype)
        want = oatt.decode_attention(q, u.keys(), u.values())
        worst = max(worst, np.max(np.abs(out[b, h * G:(h + 1) * G] - want)))
    print(f"llama3-8b layer attention max-abs error {worst:.3e}")
    assert worst < ATOL
    assert np.all(np.isfinite(out))
