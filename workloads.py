"""Seeded synthetic inputs for the RateQuant hot path.

This module only draws random numbers and names shapes. It holds none of the
method's arithmetic (no quantization, allocation, packing or attention): the
oracle and the HIP library both receive their inputs from here.

Distributions follow the workloads the paper evaluates on (Sec. 4 setup;
Appendix "Implementation Details"): per-head KV activations of Llama-3 and
Qwen3 shaped models, head_dim 128.  The real activations (WikiText-2 through
the real checkpoints) are not available; these synthetic tensors stand in
for them:

* keys  K = N(0,1) * f_c, with one outlier factor f_c ~ lognormal(0,1) per
  (layer, kv-head, channel), shared by every batch entry and token;
* values V = N(0,1); decode queries q = N(0,1);
* head-importance weights w ~ lognormal(0, sigma) and per-component
  distortion parameters beta ~ U(3.6, 5.3) for the allocator (the range of
  calibrated beta values the paper reports for KIVI, QuaRot and TurboQuant,
  Appendix "Distortion Model Parameters").

Seeds 42, 123 and 2026 are the paper's seeds (Appendix "Multi-Seed
Reliability").
"""
from __future__ import annotations

import dataclasses
import numpy as np

HEAD_DIM = 128
SEEDS = (42, 123, 2026)

KIVI, QUAROT, TURBO, RTN, KIVI_RTN = 0, 1, 2, 3, 4
F16, BF16 = 0, 1


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    family: int
    dtype: int
    n_layers: int
    batch: int
    n_kv_heads: int
    n_q_heads: int
    context: int
    residual: int
    bit_set: tuple          # allowed bit-widths (bmin..bmax)
    avg_bits: float
    w_sigma: float          # lognormal sigma of head weights
    alpha_kv: tuple         # planted alpha for (K, V) components
    fixed_bits: tuple = ()  # explicit per-head bits (same for K and V)

    @property
    def n_comp(self):
        return 2 * self.n_layers * self.n_kv_heads

    @property
    def group(self):
        return self.n_q_heads // self.n_kv_heads


# Single-layer correctness case: batch 1, 8 KV heads, 4 query heads per KV
# head, 1024 cached tokens, fp16, KIVI g32 with a 32-token residual window,
# bits [4,2,2,3,2,2,3,2] for K and V alike.
SMALL = Workload("kivi-1L-b1-t1024-fp16", KIVI, F16, 1, 1, 8, 32, 1024, 32,
                 (2, 3, 4), 2.5, 0.5, (1.0, 1.0), (4, 2, 2, 3, 2, 2, 3, 2))
# Llama-3-8B shaped KV, KIVI g32, bits {1..4} at 2.5 average.
LLAMA3_8B = Workload("llama3-8b-kv-b16-t8192-kivi-2.5b", KIVI, BF16, 32, 16,
                     8, 32, 8192, 32, (1, 2, 3, 4), 2.5, 0.5, (1.0, 1.0))
# Qwen3-8B shaped KV, QuaRot (Hadamard + symmetric per-token), bits {2..6}
# at 4.0 average.
QWEN3_8B = Workload("qwen3-8b-kv-b8-t32768-quarot-4b", QUAROT, BF16, 36, 8, 8,
                    32, 32768, 0, (2, 3, 4, 5, 6), 4.0, 0.76, (13.18, 13.04))
# Qwen3-8B shaped KV, per-token symmetric RTN (QuaRot's quantizer without the
# rotation; the paper's weakest base quantizer, run on Qwen3-8B at 3.5 and
# 4.0 bits), bits {2..6} at 4.0 average; the paper gives no RTN alpha, so
# QuaRot's planted values stand in.
QWEN3_8B_RTN = Workload("qwen3-8b-kv-b8-t32768-rtn-4b", RTN, BF16, 36, 8, 8,
                        32, 32768, 0, (2, 3, 4, 5, 6), 4.0, 0.76,
                        (13.18, 13.04))
# Llama-3-70B shaped KV, TurboQuant-style rotation + codebook, bits {2,3,4}
# at 3.0 average.
LLAMA3_70B = Workload("llama3-70b-kv-b4-t32768-turbo-3b", TURBO, BF16, 80, 4,
                      8, 64, 32768, 0, (2, 3, 4), 3.0, 0.74, (1.51, 1.50))
# Qwen3-32B shaped long context, KIVI g32 with a 128-token residual window,
# bits {1..4} at 2.0 average.
QWEN3_32B = Workload("qwen3-32b-kv-b1-t131072-kivi-2b", KIVI, BF16, 64, 1, 8,
                     64, 131072, 128, (1, 2, 3, 4), 2.0, 0.81, (17.87, 4.65))
# Llama-3-8B shaped KV with a base quantizer per side (K/V separation,
# Sec. 3.4): KIVI keys, RTN per-token values, bits {2,3,4} at 3.0 average
# (RTN needs two bits or more, so the set starts at 2 for both sides).
LLAMA3_8B_MIXED = Workload("llama3-8b-kv-b16-t8192-kivi-rtn-3b", KIVI_RTN,
                           BF16, 32, 16, 8, 32, 8192, 32, (2, 3, 4), 3.0, 0.5,
                           (1.0, 1.0))

WORKLOADS = {w.name: w for w in (SMALL, LLAMA3_8B, QWEN3_8B, LLAMA3_70B,
                                 QWEN3_32B, QWEN3_8B_RTN, LLAMA3_8B_MIXED)}


def _rng(seed, *stream):
    return np.random.default_rng([seed, *stream])


def key_outlier_factors(seed, n_layers, n_kv_heads, d=HEAD_DIM):
    """f[l][h][c] ~ lognormal(0, 1): per-channel key scale."""
    return _rng(seed, 1).lognormal(0.0, 1.0, size=(n_layers, n_kv_heads, d))


def allocation_inputs(wl: Workload, seed=42):
    """(w, alpha, beta) for the 2*L*H components, ordered (l, h, K|V)."""
    r = _rng(seed, 2)
    n = wl.n_comp
    w = r.lognormal(0.0, wl.w_sigma, size=n)
    beta = r.uniform(3.6, 5.3, size=n)
    alpha = np.tile(np.asarray(wl.alpha_kv, dtype=np.float64), n // 2)
    return w, alpha, beta


def planted_curves(n_comp, bits, seed=42, noise_sigma=0.0):
    """D(b) = alpha * beta^-b with beta ~ U(3.6, 5.3), alpha ~ lognormal,
    optionally times lognormal(0, noise_sigma) noise.  Returns
    (D[n_comp][n_bits], alpha, beta)."""
    r = _rng(seed, 3)
    beta = r.uniform(3.6, 5.3, size=n_comp)
    alpha = r.lognormal(0.0, 1.0, size=n_comp)
    b = np.asarray(bits, dtype=np.float64)
    D = alpha[:, None] * beta[:, None] ** (-b[None, :])
    if noise_sigma > 0:
        D = D * r.lognormal(0.0, noise_sigma, size=D.shape)
    return D, alpha, beta


# ---------------------------------------------------------------- CPU tensors
def bits16_from_f32(x, dtype):
    """Round float32 values to the 16-bit storage type and return the raw
    uint16 bit patterns (RNE; this is input preparation, done by numpy's /
    a plain bit recipe, not by the method)."""
    x = np.asarray(x, dtype=np.float32)
    if dtype == F16:
        return x.astype(np.float16).view(np.uint16)
    # finite inputs only: u + 0x8000 stays below 2^32 for every finite x
    u = np.ascontiguousarray(x).view(np.uint32)
    r = (u >> 16) & 1
    r += 0x7FFF
    r += u
    r >>= 16
    return r.astype(np.uint16)


def kv_cpu(wl: Workload, layer, batch_idx, n_tokens, seed=42, token0=0):
    """K, V of one (layer, batch entry) for all KV heads:
    uint16 bit patterns of shape [H][n_tokens][128] each (CPU path, small
    sizes only).  Tokens token0 .. token0+n_tokens-1 of the stream."""
    f = key_outlier_factors(seed, wl.n_layers, wl.n_kv_heads)[layer]
    r = _rng(seed, 4, layer, batch_idx, token0)
    k = r.standard_normal((wl.n_kv_heads, n_tokens, HEAD_DIM)) * f[:, None, :]
    v = r.standard_normal((wl.n_kv_heads, n_tokens, HEAD_DIM))
    return bits16_from_f32(k, wl.dtype), bits16_from_f32(v, wl.dtype)


def q_cpu(wl: Workload, layer, seed=42, step=0):
    """Decode queries [batch][Hq][128] as uint16 bit patterns."""
    r = _rng(seed, 5, layer, step)
    q = r.standard_normal((wl.batch, wl.n_q_heads, HEAD_DIM))
    return bits16_from_f32(q, wl.dtype)


def calib_cpu(n_comp, n_tokens, dtype, seed=42, key_outliers=True):
    """Calibration vectors x[n_comp][n_tokens][128] (uint16 bits): the first
    half are key components (outlier-scaled), the second half values."""
    r = _rng(seed, 6)
    x = r.standard_normal((n_comp, n_tokens, HEAD_DIM))
    if key_outliers:
        f = r.lognormal(0.0, 1.0, size=(n_comp, 1, HEAD_DIM))
        x[: n_comp // 2] *= f[: n_comp // 2]
    return bits16_from_f32(x, dtype)


def turbo_rotation(seed, layer, head, d=HEAD_DIM):
    """Seeded random rotation of one (layer, kv-head) for the TurboQuant
    quantizer: a Haar-distributed orthogonal matrix (QR of a Gaussian matrix,
    the signs of R's diagonal folded into Q), rounded to bf16.  Returns the
    uint16 bf16 bit patterns [d][d], row-major, used as y = R x."""
    g = _rng(seed, 7, layer, head).standard_normal((d, d))
    q, r = np.linalg.qr(g)
    q = q * np.sign(np.diag(r))[None, :]
    return bits16_from_f32(q.astype(np.float32), BF16)


def turbo_rotations(wl: Workload, seed=42):
    """Rotations of every (layer, kv-head): uint16 [L][H][128][128]."""
    return np.stack([np.stack([turbo_rotation(seed, l, h)
                               for h in range(wl.n_kv_heads)])
                     for l in range(wl.n_layers)])


def u16_to_f32(bits, dtype):
    """Exact widening of 16-bit patterns to float32."""
    bits = np.asarray(bits, dtype=np.uint16)
    if dtype == F16:
        return bits.view(np.float16).astype(np.float32)
    return (bits.astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------- GPU tensors
def torch_dtype(dtype):
    import torch
    return torch.float16 if dtype == F16 else torch.bfloat16


def kv_device(wl: Workload, layer, seed=42, n_tokens=None, device="cuda"):
    """K, V of one layer, shape [B][H][T][128], generated on the device by a
    seeded torch generator (large sizes).  Returns torch tensors."""
    import torch
    T = wl.context if n_tokens is None else n_tokens
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1000003 + layer * 7919 + 17)
    f = torch.from_numpy(
        key_outlier_factors(seed, wl.n_layers, wl.n_kv_heads)[layer]
    ).to(device=device, dtype=torch.float32)
    shape = (wl.batch, wl.n_kv_heads, T, HEAD_DIM)
    td = torch_dtype(wl.dtype)
    k = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    k.mul_(f[None, :, None, :])
    k = k.to(td)
    v = torch.randn(shape, generator=g, device=device,
                    dtype=torch.float32).to(td)
    return k, v


def q_device(wl: Workload, layer, seed=42, step=0, device="cuda"):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1000003 + layer * 7919 + 31 + step * 104729)
    q = torch.randn((wl.batch, wl.n_q_heads, HEAD_DIM), generator=g,
                    device=device, dtype=torch.float32)
    return q.to(torch_dtype(wl.dtype))


def haar_rotations(seed, n, d=HEAD_DIM):
    """n seeded Haar-random orthogonal d x d matrices (float64): QR of a
    Gaussian matrix with the sign of diag(R) fixed positive."""
    r = _rng(seed, 7)
    out = np.empty((n, d, d))
    for i in range(n):
        a = r.standard_normal((d, d))
        qm, rm = np.linalg.qr(a)
        out[i] = qm * np.sign(np.diag(rm))[None, :]
    return out
