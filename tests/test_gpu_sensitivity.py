"""GPU parity of the Stage-1 sensitivity reduction (rq_sensitivity) with
the oracle on the same seeded gradients: fp64 sums, relative 1e-12."""
import numpy as np
import pytest

import paper_2605_06675_amd as rq
from oracle import sensitivity as osens

pytestmark = pytest.mark.gpu

RTOL = 1e-12


def _grads(S, n, T, seed):
    rng = np.random.default_rng(seed)
    # heavy-tailed per-component scales, as gradient norms are across heads
    scale = rng.lognormal(0.0, 1.5, size=(1, n, 1, 1))
    return (rng.standard_normal((S, n, T, 128)) * scale * 1e-3).astype(np.float32)


def _run(gdtype, g32):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    tdt = {rq.RQ_F32: torch.float32, rq.RQ_F16: torch.float16,
           rq.RQ_BF16: torch.bfloat16}[gdtype]
    dev = torch.from_numpy(g32).to("cuda").to(tdt).contiguous()
    exact = dev.float().cpu().numpy()       # the values the kernel reads
    w = rq.rq_sensitivity(gdtype, dev)
    torch.cuda.synchronize()
    return w, osens.sensitivity(exact)


@pytest.mark.parametrize("gdtype", [rq.RQ_F32, rq.RQ_F16, rq.RQ_BF16])
def test_small_every_dtype(gdtype):
    print(f"sensitivity small dtype {gdtype}", flush=True)
    g = _grads(3, 5, 96, 1)
    if gdtype == rq.RQ_F16:
        g = g * 1e3                          # keep fp16 values normal
    w, want = _run(gdtype, g)
    np.testing.assert_allclose(w, want, rtol=RTOL)


@pytest.mark.parametrize("T", [1, 1000])
def test_ragged_chunks(T):
    # T=1: one short slab; T=1000: three full chunks and a ragged fourth
    print(f"sensitivity ragged T={T}", flush=True)
    w, want = _run(rq.RQ_F32, _grads(2, 3, T, 2))
    np.testing.assert_allclose(w, want, rtol=RTOL)


def test_calibration_sized_with_cap_and_allocation():
    # 16 sequences x 512 tokens (the paper's calibration set) for 64
    # components; then the cap and an allocation on the result
    print("sensitivity 16 x 64 x 512", flush=True)
    w, want = _run(rq.RQ_F32, _grads(16, 64, 512, 3))
    np.testing.assert_allclose(w, want, rtol=RTOL)
    wc = rq.rq_cap_weights(w)
    np.testing.assert_allclose(wc, osens.cap_weights(want), rtol=RTOL)
    beta = np.random.default_rng(4).uniform(3.6, 5.3, size=64)
    bits, _, _ = rq.rq_allocate_bits(wc, np.ones(64), beta, 3.0, 2, 6)
    assert bits.sum() == 192
