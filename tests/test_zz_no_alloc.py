"""rq_decode_attention_static (the entry point that allocates nothing: its
counters and partials live in the library's static device scratch) against
rq_decode_attention with a caller workspace, through the C-ABI: two calls in
a row on the same GPU, the second on a smaller cache, each within the
attention tolerance of the workspace call and of the oracle; and a shape
whose partials exceed the scratch is rejected before any launch."""
import numpy as np
import pytest

import paper_2605_06675_amd as rq
import workloads
from oracle import attention as oatt
from tests import gpu_helpers as gh
from tests import test_gpu_parity as gp

pytestmark = pytest.mark.gpu


def _run(family, dtype, H, G, T, R, bits, batch, seed):
    import torch
    kvc, ks, vs, _ = gp._build(family, dtype, H, G, T, R, bits, batch=batch,
                               seed=seed)
    units = gp._check_cache(family, dtype, kvc, ks, vs, bits, R, batch, H, T)
    q16 = workloads.bits16_from_f32(
        np.random.default_rng(seed).standard_normal((batch, H * G, 128)), dtype)
    q = gh.dev(q16, dtype)
    ref = kvc.attention(0, q)
    out = torch.full_like(ref, float("nan"))
    kvc.attention_static(0, q, out)
    torch.cuda.synchronize()
    ref, out = ref.cpu().numpy(), out.cpu().numpy()
    assert np.all(np.isfinite(out))
    diff = float(np.max(np.abs(out - ref)))
    worst = 0.0
    for (b, h), u in units.items():
        qq = workloads.u16_to_f32(q16[b, h * G:(h + 1) * G], dtype)
        want = oatt.decode_attention(qq, u.keys(), u.values())
        worst = max(worst, float(np.max(np.abs(out[b, h * G:(h + 1) * G] - want))))
    print(f"static vs workspace {diff:.2e}, static vs oracle {worst:.2e}")
    assert diff < gp.ATOL
    assert worst < gp.ATOL


def test_static_scratch_two_calls_second_smaller():
    # first: 4 x 8 units of 2080 tokens (several workgroups per unit, a
    # window); second: 2 x 4 units of 300 tokens in another family
    bits1 = np.array([[[1 + h % 4, 4 - h % 4] for h in range(8)]])
    _run(workloads.KIVI, workloads.BF16, 8, 4, 2080, 32, bits1, 4, seed=3)
    bits2 = np.array([[[2, 3], [4, 2], [3, 3], [5, 2]]])
    _run(workloads.QUAROT, workloads.F16, 4, 2, 300, 16, bits2, 2, seed=4)


def test_static_scratch_rejects_oversized_partials():
    import torch
    # 64 x 32 units with 16 query heads each: the partials exceed 7 MiB
    bits = np.full((1, 32, 2), 2, dtype=np.int8)
    kvc = rq.KVCache(rq.RQ_KIVI, rq.RQ_BF16, 1, 64, 32, 512, 4096, 0, bits)
    kvc.n_tokens[0] = 4096
    q = torch.zeros((64, 512, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((64, 512, 128), dtype=torch.float32, device="cuda")
    with pytest.raises(rq.RQError) as e:
        kvc.attention_static(0, q, out)
    assert e.value.status == rq.RQ_ESMALLWS
