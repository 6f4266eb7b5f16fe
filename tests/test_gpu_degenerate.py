"""GPU parity on the degenerate inputs the quantizers special-case, for every
family: all-zero tokens and groups (scale or norm 0), constant rows (KIVI's
min-max range 0), single-channel spikes, and bf16 values beyond the fp16
range (the fp16 metadata saturates at 65504), and queries far above and
below unit scale.  Codes, metadata and the window must match the oracle
(TurboQuant codes by its near-threshold rule); attention must match it
everywhere, to 1e-2 at unit scale and in proportion beyond."""
import numpy as np
import pytest

import paper_2605_06675_amd as rq
import workloads
from oracle import cache as ocache
from tests import gpu_helpers as gh
from tests import test_gpu_parity as gp
from tests import test_gpu_turbo as gt

pytestmark = pytest.mark.gpu

H, G, T, R, BATCH = 4, 4, 224, 32, 2


def _data(seed, scale=1.0):
    """[B][H][T][128] float32: every 7th token zero, then constant rows,
    single spikes, whole-zero 32-token blocks for one head, Gaussian rest."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((BATCH, H, T, 128))
    t = np.arange(T)
    x[:, :, t % 7 == 0] = 0.0
    x[:, :, t % 7 == 1] = 0.5
    spike = t % 7 == 2
    x[:, :, spike] = 0.0
    x[:, :, spike, 17] = 12.0
    x[:, 1, 32:64] = 0.0                      # one block all zero (keys: s = 0)
    x[:, 2, 64:96, :40] = -3.0                # constant channels over a block
    return x * scale


def _fill(family, dtype, bits, kf, vf, rotation=None):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    ks = [workloads.bits16_from_f32(kf[b], dtype) for b in range(BATCH)]
    vs = [workloads.bits16_from_f32(vf[b], dtype) for b in range(BATCH)]
    kvc = rq.KVCache(family, dtype, 1, BATCH, H, H * G, T, R, bits,
                     rotation=rotation)
    K, V = gh.dev(np.stack(ks), dtype), gh.dev(np.stack(vs), dtype)
    kvc.append(0, K[:, :, :150].contiguous(), V[:, :, :150].contiguous())
    kvc.append(0, K[:, :, 150:].contiguous(), V[:, :, 150:].contiguous())
    torch.cuda.synchronize()
    return kvc, ks, vs


@pytest.mark.parametrize("family,bits", [
    (workloads.KIVI, [[1, 4], [2, 3], [3, 2], [8, 1]]),
    (workloads.QUAROT, [[2, 4], [3, 3], [4, 2], [8, 5]]),
    (workloads.RTN, [[2, 4], [3, 3], [4, 2], [8, 5]]),
    (workloads.KIVI_RTN, [[1, 4], [2, 3], [3, 2], [8, 2]])],
    ids=["kivi", "quarot", "rtn", "kivi_rtn"])
@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
def test_degenerate_affine_families(family, bits, dtype):
    print(f"degenerate family {family} dtype {dtype}", flush=True)
    bits = np.array([bits])
    kvc, ks, vs = _fill(family, dtype, bits, _data(1), _data(2))
    units = gp._check_cache(family, dtype, kvc, ks, vs, bits, R, BATCH, H, T)
    gp._check_attention(kvc, units, dtype, BATCH, H, G)


@pytest.mark.parametrize("family", [workloads.KIVI, workloads.QUAROT,
                                    workloads.RTN, workloads.KIVI_RTN],
                         ids=["kivi", "quarot", "rtn", "kivi_rtn"])
def test_saturated_metadata_bf16(family):
    # |x| up to ~1e7: scales and zero points saturate at the fp16 maximum
    print(f"saturated metadata family {family}", flush=True)
    bits = np.array([[[2, 3], [3, 2], [4, 4], [5, 6]]])
    kvc, ks, vs = _fill(family, workloads.BF16, bits, _data(3, 2.0e5), _data(4, 2.0e5))
    units = gp._check_cache(family, workloads.BF16, kvc, ks, vs, bits, R, BATCH, H, T)
    gp._check_attention(kvc, units, workloads.BF16, BATCH, H, G)


@pytest.mark.parametrize("q_mult", [1.0e6, 1.0e-6], ids=["q1e6", "q1e-6"])
@pytest.mark.parametrize("family", [workloads.KIVI, workloads.QUAROT,
                                    workloads.RTN, workloads.KIVI_RTN],
                         ids=["kivi", "quarot", "rtn", "kivi_rtn"])
def test_large_values_and_queries(family, q_mult):
    # value scales near the fp16 maximum (probability x scale beyond the
    # fp16 range) and queries whose scaled elements leave it (q1e6) or
    # underflow it (q1e-6)
    print(f"large values family {family} q x {q_mult:g}", flush=True)
    bits = np.array([[[2, 2], [3, 2], [4, 3], [8, 5]]])
    rng = np.random.default_rng(11)
    kf = rng.standard_normal((BATCH, H, T, 128))
    vf = rng.standard_normal((BATCH, H, T, 128)) * 3.0e4
    kvc, ks, vs = _fill(family, workloads.BF16, bits, kf, vf)
    units = gp._check_cache(family, workloads.BF16, kvc, ks, vs, bits, R, BATCH, H, T)
    gp._check_attention(kvc, units, workloads.BF16, BATCH, H, G, q_mult=q_mult)


def test_degenerate_turbo():
    print("degenerate turbo", flush=True)
    dtype = workloads.BF16
    bits = np.array([[[1, 4], [2, 3], [3, 2], [4, 4]]])
    r16, rf = gt._rotations(1, H)
    kvc, ks, vs = _fill(workloads.TURBO, dtype, bits, _data(5), _data(6),
                        rotation=gh.dev(r16, workloads.BF16))
    units = gt._check(dtype, kvc, ks, vs, rf[0], bits, R, BATCH, H)
    gt._attention(kvc, units, dtype, BATCH, H, G)


@pytest.mark.parametrize("q_mult", [1.0e6, 1.0e-6], ids=["q1e6", "q1e-6"])
def test_large_values_and_queries_turbo(q_mult):
    # norms near the fp16 maximum (probability x norm / sqrt(128) beyond
    # the fp16 range) and queries far from unit scale; widths 1..8
    print(f"large values turbo q x {q_mult:g}", flush=True)
    dtype = workloads.BF16
    bits = np.array([[[1, 6], [3, 8], [5, 2], [7, 4]]])
    rng = np.random.default_rng(12)
    kf = rng.standard_normal((BATCH, H, T, 128))
    vf = rng.standard_normal((BATCH, H, T, 128)) * 5.0e3
    r16, rf = gt._rotations(1, H)
    kvc, ks, vs = _fill(workloads.TURBO, dtype, bits, kf, vf,
                        rotation=gh.dev(r16, workloads.BF16))
    units = gt._check(dtype, kvc, ks, vs, rf[0], bits, R, BATCH, H)
    gt._attention(kvc, units, dtype, BATCH, H, G, q_mult=q_mult)
