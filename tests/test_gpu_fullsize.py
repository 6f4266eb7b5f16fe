"""GPU parity at full size: one layer of each long-context workload, filled
the way the benchmark fills it (prefill of T - s tokens, then s single-token
appends, s = 64 for the long-context KIVI workload and 1 otherwise), then
decode attention over all T tokens; sampled (batch, kv-head) units, one of
every width pair of the layer among them, checked against the oracle (codes, metadata and window bit-exact, TurboQuant codes by
its near-threshold rule; attention within 1e-2 max-abs)."""
import numpy as np
import pytest

import paper_2605_06675_amd as rq
import workloads
from oracle import attention as oatt
from oracle import cache as ocache
from oracle import quant as oquant
from tests import gpu_helpers as gh
from tests import test_gpu_turbo as gt

pytestmark = pytest.mark.gpu

ATOL = 1e-2
DECODE_STEPS = {workloads.QWEN3_32B.name: 64}


def _turbo_unit(lay, bufs, b, h, u, k, v, k16, v16, Rh, R):
    """Metadata and window exact; codes exact away from thresholds."""
    codes_u8, meta_u8, resid_u16 = bufs
    nq, bk, bv = u.nq, u.bk, u.bv
    for kind, want in ((0, u.k_meta), (1, u.v_meta)):
        got = lay.meta(meta_u8, 0, b, h, kind, nq // 32)
        np.testing.assert_array_equal(got.view(np.uint16),
                                      np.asarray(want).view(np.uint16))
    gk = ocache.unpack_keys(lay.k_words(codes_u8, 0, b, h, nq), bk)
    gv = ocache.unpack_values(lay.v_words(codes_u8, 0, b, h, nq // 32), bv)
    mism = gt._compare_codes(gk, u.k_codes, u.k_t, bk,
                             gt._eps(k[:nq], Rh, oquant.turbo_norm(k[:nq]), u.k_t),
                             f"K b{b} h{h}")
    mism += gt._compare_codes(gv, u.v_codes, u.v_t, bv,
                              gt._eps(v[:nq], Rh, oquant.turbo_norm(v[:nq]), u.v_t),
                              f"V b{b} h{h}")
    for kind, src in ((0, k16), (1, v16)):
        ring = lay.ring(resid_u16, 0, b, h, kind)
        for t in range(nq, u.T):
            np.testing.assert_array_equal(ring[ocache.ring_slot(t, R)], src[t])
    return mism, 2 * nq * 128


@pytest.mark.parametrize("wl", [workloads.QWEN3_8B, workloads.QWEN3_8B_RTN,
                                workloads.LLAMA3_70B, workloads.QWEN3_32B],
                         ids=lambda w: w.name)
def test_full_size_layer_sampled(wl):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    print(f"full-size layer {wl.name}", flush=True)
    L, H, B, T = wl.n_layers, wl.n_kv_heads, wl.batch, wl.context
    lo, hi = min(wl.bit_set), max(wl.bit_set)
    w, a, be = workloads.allocation_inputs(wl)
    alloc_bits, _, _ = rq.rq_allocate_bits(w, a, be, wl.avg_bits, lo, hi)
    bits = alloc_bits.reshape(L, H, 2)[:1]
    turbo = wl.family == workloads.TURBO
    rot, Rf = None, None
    if turbo:
        r16 = np.stack([[workloads.turbo_rotation(42, 0, h) for h in range(H)]])
        rot = gh.dev(r16, workloads.BF16)
        Rf = workloads.u16_to_f32(r16[0], workloads.BF16).astype(np.float64)
    steps = DECODE_STEPS.get(wl.name, 1)
    T0 = T - steps
    K, V = workloads.kv_device(wl, 0)
    kvc = rq.KVCache(wl.family, wl.dtype, 1, B, H, wl.n_q_heads, T,
                     wl.residual, bits, rotation=rot)
    kvc.append(0, K[:, :, :T0].contiguous(), V[:, :, :T0].contiguous())
    for s in range(steps):
        t = T0 + s
        kvc.append(0, K[:, :, t:t + 1].contiguous(), V[:, :, t:t + 1].contiguous())
    qd = workloads.q_device(wl, 0)
    out = kvc.attention(0, qd)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    assert np.all(np.isfinite(out))
    q16 = gh.host_bits(qd)
    lay = gh.Layout(wl.family, 1, B, H, T, wl.residual, bits)
    bufs = gh.read_buffers(kvc)
    G = wl.group
    worst, mism, total = 0.0, 0, 0
    # three fixed units, plus one unit of every (K, V) width pair the
    # allocation gave this layer
    first_of_pair = {}
    for h in range(H):
        first_of_pair.setdefault(tuple(int(x) for x in bits[0, h]), h)
    units = {(0, 0), (B // 2, 3), (B - 1, H - 1)}
    units |= {(h % B, h) for h in first_of_pair.values()}
    for (b, h) in sorted(units):
        k16, v16 = gh.host_bits(K[b, h]), gh.host_bits(V[b, h])
        k = workloads.u16_to_f32(k16, wl.dtype)
        v = workloads.u16_to_f32(v16, wl.dtype)
        u = ocache.Unit(wl.family, k, v, int(bits[0, h, 0]), int(bits[0, h, 1]),
                        wl.residual, rotation=Rf[h] if turbo else None)
        if turbo:
            m, n = _turbo_unit(lay, bufs, b, h, u, k, v, k16, v16, Rf[h],
                               wl.residual)
            mism, total = mism + m, total + n
        else:
            gh.compare_unit(lay, bufs, 0, b, h, u, k16, v16)
        q = workloads.u16_to_f32(q16[b, h * G:(h + 1) * G], wl.dtype)
        want = oatt.decode_attention(q, u.keys(), u.values())
        err = np.max(np.abs(out[b, h * G:(h + 1) * G] - want))
        print(f"  unit b{b} h{h} bits {bits[0, h].tolist()}: attention err {err:.2e}",
              flush=True)
        worst = max(worst, err)
    if turbo:
        print(f"  codes {total}, adjacent near-threshold differences {mism}")
        assert mism <= max(2, total // 1000)
    assert worst < ATOL
