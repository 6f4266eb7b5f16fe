"""Base quantizers (oracle).

The paper treats the base quantizer as a black box with a calibrated
distortion curve (Sec. 3.4) and names three: KIVI (keys grouped per channel
across tokens, values per token), QuaRot (a Hadamard rotation, then
symmetric per-token quantization) and TurboQuant (a random rotation, then a
per-coordinate codebook) -- Sec. 2, Appendix "Implementation Details" and
"Quantizer Implementation".  It gives no rounding rules; the ones below are
this library's readings (each is listed in the design notes) and both the
oracle and the GPU kernels follow them bit for bit wherever a floating-point
decision yields an integer code:

* inputs are fp16 or bf16, widened exactly to fp32;
* metadata (scale, zero, norm) is fp16, rounded to nearest-even from an fp32
  value and saturated at +-65504;
* every arithmetic step that decides a code is one correctly-rounded fp32
  operation (no fused multiply-add), and rint is round-half-to-even.

Dequantization (used for attention and for the distortion sweep) is exact
real arithmetic on the stored codes and metadata, evaluated in fp64.
"""
import math

import numpy as np

from . import fmt

F32 = np.float32
D = 128
INV_SQRT_D_F32 = F32(1.0 / math.sqrt(128.0))


# --------------------------------------------------------------------- KIVI
def kivi_groups(x, b):
    """Asymmetric min/max quantization of groups along the last axis.

    x: float32[..., g].  Returns (codes int64[..., g], s fp16[...], z fp16[...]).
      z = fp16(min);  s = fp16(max(max - z, 0) / (2^b - 1));
      code = rint(clamp((x - z) * (1/s), 0, 2^b - 1)),  all codes 0 if s == 0.
    """
    x = np.asarray(x, dtype=F32)
    qmax = F32((1 << b) - 1)
    mn = x.min(axis=-1)
    mx = x.max(axis=-1)
    z = fmt.f16_sat(mn)
    zf = z.astype(F32)
    rng = np.maximum(mx - zf, F32(0))            # fp32 subtraction
    s = fmt.f16_sat(rng / qmax)                  # fp32 division, then fp16
    sf = s.astype(F32)
    valid = sf != 0
    inv = np.where(valid, F32(1) / np.where(valid, sf, F32(1)), F32(0))
    r = (x - zf[..., None]) * inv[..., None]     # two fp32 roundings
    u = np.rint(np.clip(r, F32(0), qmax)).astype(np.int64)
    u = np.where(valid[..., None], u, 0)
    return u, s, z


def kivi_dequant(u, s, z):
    """x_hat = u * s + z  (fp64)."""
    return (np.asarray(u, dtype=np.float64) * np.asarray(s, np.float64)[..., None]
            + np.asarray(z, np.float64)[..., None])


def kivi_quant_keys(x, b):
    """Keys of one (layer, batch, kv-head): x float32[T][128], T % 32 == 0.
    Groups: one channel across 32 consecutive tokens.
    Returns codes[T][128], s[T/32][128], z[T/32][128]."""
    T = x.shape[0]
    assert T % 32 == 0 and x.shape[1] == D
    g = x.reshape(T // 32, 32, D).transpose(0, 2, 1)     # [blk][c][32 tok]
    u, s, z = kivi_groups(g, b)
    return u.transpose(0, 2, 1).reshape(T, D), s, z


def kivi_dequant_keys(u, s, z):
    T = u.shape[0]
    g = u.reshape(T // 32, 32, D).transpose(0, 2, 1)
    return kivi_dequant(g, s, z).transpose(0, 2, 1).reshape(T, D)


def kivi_quant_values(x, b):
    """Values: groups of 32 consecutive channels of one token.
    Returns codes[T][128], s[T][4], z[T][4]."""
    T = x.shape[0]
    u, s, z = kivi_groups(x.reshape(T, 4, 32), b)
    return u.reshape(T, D), s, z


def kivi_dequant_values(u, s, z):
    T = u.shape[0]
    return kivi_dequant(u.reshape(T, 4, 32), s, z).reshape(T, D)


# ------------------------------------------------------------------- QuaRot
def fwht_f32(x):
    """Unnormalised Walsh-Hadamard transform along the last axis (length
    128, Sylvester order) in fp32 with a fixed butterfly order: for
    h = 1, 2, 4, ..., 64, pairs (i, i+h) inside blocks of 2h become
    (a + b, a - b)."""
    v = np.array(x, dtype=F32)
    n = v.shape[-1]
    assert n == D
    lead = v.shape[:-1]
    h = 1
    while h < n:
        w = v.reshape(lead + (n // (2 * h), 2, h))
        a = w[..., 0, :].copy()
        bb = w[..., 1, :].copy()
        w[..., 0, :] = a + bb
        w[..., 1, :] = a - bb
        v = w.reshape(lead + (n,))
        h *= 2
    return v


def hadamard(n=D):
    """Sylvester Hadamard matrix H_n (entries +-1, H H^T = n I)."""
    H = np.array([[1.0]])
    while H.shape[0] < n:
        H = np.block([[H, H], [H, -H]])
    return H


def quarot_rotate(x):
    """y = fp32(fwht(x) * fp32(1/sqrt(128)))."""
    return fwht_f32(x) * INV_SQRT_D_F32


def quarot_quant(x, b):
    """Symmetric per-token quantization of the rotated vector.
    x float32[T][128] -> codes[T][128] (offset binary), s fp16[T].
      y = rotate(x);  a = max|y|;  s = fp16(a / (2^(b-1) - 1));
      q = rint(clamp(y * (1/s), -qm, qm));  code = q + 2^(b-1)."""
    if b < 2:
        raise ValueError("symmetric quantizer needs b >= 2")
    y = quarot_rotate(x)
    qm = F32((1 << (b - 1)) - 1)
    a = np.max(np.abs(y), axis=-1)
    s = fmt.f16_sat(a / qm)
    sf = s.astype(F32)
    valid = sf != 0
    inv = np.where(valid, F32(1) / np.where(valid, sf, F32(1)), F32(0))
    q = np.rint(np.clip(y * inv[..., None], -qm, qm)).astype(np.int64)
    q = np.where(valid[..., None], q, 0)
    return q + (1 << (b - 1)), s


def quarot_dequant(u, s, b):
    """x_hat = (1/sqrt(128)) H ((u - 2^(b-1)) s)  (fp64, H symmetric)."""
    yhat = (np.asarray(u, np.float64) - (1 << (b - 1))) * np.asarray(
        s, np.float64)[..., None]
    return yhat @ hadamard() / math.sqrt(D)
