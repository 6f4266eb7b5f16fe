"""Distortion sweep (oracle).

Stage 2 of Alg. 1 measures the MSE of the base quantizer at several
bit-widths before fitting D(b) = alpha * beta^-b.  Here
    D_i(b) = mean over tokens and channels of (x - x_hat_b)^2
for component i (its calibration vectors x[T][128]), with x_hat_b the
quantize -> dequantize round trip at b bits, measured in the original
(unrotated) domain, accumulated in fp64.  Key components use the key
grouping of their family, value components the value grouping.
"""
import numpy as np

from . import quant

KIVI, QUAROT, TURBO, RTN, KIVI_RTN = 0, 1, 2, 3, 4


def roundtrip(family, x, b, is_value, rotation=None):
    if family == KIVI_RTN:
        # the mixed family: KIVI keys, RTN values
        family = RTN if is_value else KIVI
    if family == KIVI:
        if is_value:
            u, s, z = quant.kivi_quant_values(x, b)
            return quant.kivi_dequant_values(u, s, z)
        u, s, z = quant.kivi_quant_keys(x, b)
        return quant.kivi_dequant_keys(u, s, z)
    if family == QUAROT:
        u, s = quant.quarot_quant(x, b)
        return quant.quarot_dequant(u, s, b)
    if family == RTN:
        u, s = quant.rtn_quant(x, b)
        return quant.rtn_dequant(u, s, b)
    if family == TURBO:
        u, n, _ = quant.turbo_quant(x, rotation, b)
        return quant.turbo_dequant(u, n, rotation, b)
    raise NotImplementedError(family)


def sweep(family, x, bits, is_value, rotations=None):
    """x: float32[n_comp][T][128] -> D float64[n_comp][len(bits)].
    rotations: TurboQuant's per-component rotation [n_comp][128][128]."""
    x = np.asarray(x, dtype=np.float32)
    out = np.zeros((x.shape[0], len(bits)))
    for i in range(x.shape[0]):
        xi = x[i].astype(np.float64)
        rot = None if rotations is None else rotations[i]
        for j, b in enumerate(bits):
            xh = roundtrip(family, x[i], b, is_value, rot)
            out[i, j] = np.mean((xi - xh) ** 2)
    return out
