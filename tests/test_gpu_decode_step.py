"""GPU parity of the fused decode step (rq_decode_step): per layer and
step, the flush of the block that leaves the residual window, the window
append and the decode attention in as few launches as possible.  Over steps
that cross block flushes it must leave exactly the cache that
rq_quantize_kv + rq_decode_attention leave (codes, metadata and window
bit-exact), return the same attention (to fp32 summation order), and match
the oracle (Appendix "Runtime Analysis": the decode path of the mixed-bit
cache)."""
import numpy as np
import pytest

import paper_2605_06675_amd as rq
import workloads
from tests import gpu_helpers as gh
from tests import test_gpu_parity as gp
from tests import test_gpu_turbo as gt

pytestmark = pytest.mark.gpu

H, G, B, T0, STEPS = 3, 4, 2, 290, 75


@pytest.mark.parametrize("family,R,bits,dtype", [
    (workloads.KIVI, 32, [[2, 3], [1, 4], [4, 2]], workloads.BF16),
    (workloads.QUAROT, 0, [[2, 3], [4, 2], [3, 3]], workloads.BF16),
    (workloads.RTN, 16, [[5, 2], [2, 6], [3, 3]], workloads.F16),
    (workloads.TURBO, 0, [[2, 3], [4, 2], [3, 6]], workloads.BF16),
    (workloads.KIVI_RTN, 16, [[1, 2], [3, 4], [4, 3]], workloads.F16)],
    ids=["kivi", "quarot", "rtn", "turbo", "kivi_rtn"])
def test_decode_step_equals_append_then_attention(family, R, bits, dtype):
    torch = gp._torch()
    bits = np.array([bits])
    T = T0 + STEPS
    wl = workloads.Workload("t", family, dtype, 1, B, H, H * G, T, R, (1,),
                            2.0, 0.5, (1.0, 1.0))
    ks, vs = zip(*[workloads.kv_cpu(wl, 0, b, T) for b in range(B)])
    K, V = gh.dev(np.stack(ks), dtype), gh.dev(np.stack(vs), dtype)
    rot = None
    if family == workloads.TURBO:
        r16, rf = gt._rotations(1, H)
        rot = gh.dev(r16, workloads.BF16)
    cap = ((T + 31) // 32) * 32
    fused = rq.KVCache(family, dtype, 1, B, H, H * G, cap, R, bits, rotation=rot)
    split = rq.KVCache(family, dtype, 1, B, H, H * G, cap, R, bits, rotation=rot)
    for c in (fused, split):
        c.append(0, K[:, :, :T0].contiguous(), V[:, :, :T0].contiguous())
    rng = np.random.default_rng(3)
    worst = 0.0
    print(f"decode step family {family} R {R}", flush=True)
    for s in range(STEPS):
        t = T0 + s
        k1, v1 = K[:, :, t:t + 1].contiguous(), V[:, :, t:t + 1].contiguous()
        q = gh.dev(workloads.bits16_from_f32(
            rng.standard_normal((B, H * G, 128)), dtype), dtype)
        a = fused.decode_step(0, k1, v1, q)
        split.append(0, k1, v1)
        b = split.attention(0, q)
        torch.cuda.synchronize()
        worst = max(worst, float((a - b).abs().max()))
    print(f"  fused vs split max-abs {worst:.2e}")
    assert worst < 1e-4
    assert fused.n_tokens[0] == split.n_tokens[0] == T
    for x, y in ((fused.codes, split.codes), (fused.meta, split.meta),
                 (fused.resid, split.resid)):
        assert torch.equal(x, y)
    if family == workloads.TURBO:
        units = gt._check(dtype, fused, list(ks), list(vs), rf[0], bits, R, B, H)
        gt._attention(fused, units, dtype, B, H, G)
    else:
        units = gp._check_cache(family, dtype, fused, list(ks), list(vs), bits,
                                R, B, H, T)
        gp._check_attention(fused, units, dtype, B, H, G)


def test_decode_step_validates_before_launching():
    torch = gp._torch()
    bits = np.array([[[2, 2]]])
    c = rq.KVCache(workloads.KIVI, workloads.BF16, 1, 1, 1, 4, 64, 32, bits)
    k = torch.zeros((1, 1, 1, 128), dtype=torch.bfloat16, device="cuda")
    q = torch.zeros((1, 4, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.empty((1, 4, 128), dtype=torch.float32, device="cuda")
    ws = torch.zeros(8, dtype=torch.uint8, device="cuda")   # too small
    with pytest.raises(rq.RQError):
        rq.rq_decode_step(c.desc, 0, 0, k, k, q, out, ws)
    with pytest.raises(rq.RQError):
        rq.rq_decode_step(c.desc, 0, 64, k, k, q, out, c.workspace(64))
    torch.cuda.synchronize()
    assert int(c.resid.abs().sum()) == 0 and int(c.codes.sum()) == 0
