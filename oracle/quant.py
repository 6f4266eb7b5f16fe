"""Base quantizers (oracle).

The paper treats the base quantizer as a black box with a calibrated
distortion curve (Sec. 3.4) and names three: KIVI (keys grouped per channel
across tokens, values per token), QuaRot (a Hadamard rotation, then
symmetric per-token quantization) and TurboQuant (a random rotation, then a
per-coordinate codebook) -- Sec. 2, Sec. 3.1, Appendix "Implementation
Details" and "Quantizer Implementation" -- and, as the weakest base
quantizer, plain per-token symmetric round-to-nearest (Appendix "RTN Base
Quantizer").  It gives no rounding rules; the ones below are
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
import functools
import math

import numpy as np

from . import fmt, lloydmax

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


def sym_per_token(y, b):
    """Symmetric per-token quantization of y float32[T][128] over all 128
    channels -> codes[T][128] (offset binary), s fp16[T].
      a = max|y|;  s = fp16(a / (2^(b-1) - 1));
      q = rint(clamp(y * (1/s), -qm, qm));  code = q + 2^(b-1).
    A token with s == 0 gets q = 0 everywhere."""
    if b < 2:
        raise ValueError("symmetric quantizer needs b >= 2")
    y = np.asarray(y, dtype=F32)
    qm = F32((1 << (b - 1)) - 1)
    a = np.max(np.abs(y), axis=-1)
    s = fmt.f16_sat(a / qm)
    sf = s.astype(F32)
    valid = sf != 0
    inv = np.where(valid, F32(1) / np.where(valid, sf, F32(1)), F32(0))
    q = np.rint(np.clip(y * inv[..., None], -qm, qm)).astype(np.int64)
    q = np.where(valid[..., None], q, 0)
    return q + (1 << (b - 1)), s


def quarot_quant(x, b):
    """Symmetric per-token quantization of the rotated vector:
    sym_per_token(rotate(x), b)."""
    if b < 2:
        raise ValueError("symmetric quantizer needs b >= 2")
    return sym_per_token(quarot_rotate(x), b)


def quarot_dequant(u, s, b):
    """x_hat = (1/sqrt(128)) H ((u - 2^(b-1)) s)  (fp64, H symmetric)."""
    yhat = (np.asarray(u, np.float64) - (1 << (b - 1))) * np.asarray(
        s, np.float64)[..., None]
    return yhat @ hadamard() / math.sqrt(D)


# ---------------------------------------------------------------------- RTN
# Round-to-nearest, per-token symmetric (Appendix "RTN Base Quantizer",
# Table "RTN per-token symmetric on Qwen3-8B"): QuaRot's symmetric step
# applied to the vector itself, one scale per token over its 128 channels.
def rtn_quant(x, b):
    """codes[T][128] (offset binary), s fp16[T] = sym_per_token(x, b)."""
    return sym_per_token(x, b)


def rtn_dequant(u, s, b):
    """x_hat = (u - 2^(b-1)) s  (fp64)."""
    return (np.asarray(u, np.float64) - (1 << (b - 1))) * np.asarray(
        s, np.float64)[..., None]


# --------------------------------------------------------------- TurboQuant
# A random rotation spreads each vector's energy evenly over the coordinates,
# which then follow (nearly) a Gaussian of variance |x|^2 / d; each rotated
# coordinate, normalised by |x| / sqrt(d), is quantized with the Lloyd-Max
# quantizer of N(0,1) at b bits (Sec. 2; Sec. 3.1, whose Table 6 lists that
# quantizer's MSE).  Readings:
#  * the rotation R is an input: one orthogonal matrix per (layer, kv-head),
#    given as bf16 values (the workloads draw it from the Haar measure);
#    y = R x with the exact products and sums (fp64 here);
#  * the norm is stored per token as fp16: n = fp16(fp32(sqrt(sum x^2))),
#    the sum and root taken in fp64;
#  * t = y * sqrt(128) / n (t = 0 when n == 0) and the code is the number of
#    thresholds below t, code = #{k : t > theta_k}, theta_k the fp32 midpoint
#    of Lloyd-Max centroids k and k+1 (ties to the lower code);
#  * dequantization: y_hat = c_code * n / sqrt(128), x_hat = R^T y_hat.
SQRT_D = math.sqrt(128.0)


@functools.lru_cache(maxsize=None)
def turbo_codebook(b):
    """(centroids fp64 [2^b], thresholds fp32 [2^b - 1]) of N(0,1)."""
    c = lloydmax.centroids(b)
    return c, lloydmax.thresholds_f32(c)


def turbo_norm(x):
    """fp16 norm of each row of x (float32 [T][128])."""
    n = np.sqrt(np.sum(np.asarray(x, np.float64) ** 2, axis=-1))
    return fmt.f16_sat(n.astype(np.float32))


def turbo_quant(x, R, b):
    """x float32 [T][128] (exact 16-bit values), R float64 [128][128].
    Returns (codes int64 [T][128], n fp16 [T], t float64 [T][128])."""
    x = np.asarray(x, dtype=np.float64)
    R = np.asarray(R, dtype=np.float64)
    y = x @ R.T                                   # y_t = R x_t
    n = turbo_norm(x)
    nf = n.astype(np.float64)
    safe = np.where(nf > 0, nf, 1.0)
    t = np.where(nf[:, None] > 0, y * SQRT_D / safe[:, None], 0.0)
    _, th = turbo_codebook(b)
    codes = np.sum(t[..., None] > th.astype(np.float64), axis=-1)
    return codes.astype(np.int64), n, t


def turbo_dequant(u, n, R, b):
    """x_hat [T][128] (fp64) from codes, fp16 norms and the rotation."""
    c, _ = turbo_codebook(b)
    yhat = c[np.asarray(u)] * (np.asarray(n, np.float64)[:, None] / SQRT_D)
    return yhat @ np.asarray(R, dtype=np.float64)   # x_hat_t = R^T y_hat_t


def turbo_near_threshold(t, b, eps):
    """Boolean mask of coordinates whose t lies within eps of a threshold
    (where a computation in another precision may pick the adjacent code)."""
    _, th = turbo_codebook(b)
    d = np.min(np.abs(np.asarray(t)[..., None] - th.astype(np.float64)), axis=-1)
    return d <= eps
