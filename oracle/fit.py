"""Distortion-model fit (oracle).

The paper models the MSE of a base quantizer at b bits as
D(b) = alpha * beta^-b with alpha > 0, beta > 1 (Sec. 3.1, Assumption 1) and
calibrates (alpha, beta) per quantizer by least squares on
ln D = ln alpha - b ln beta over a set of bit-widths (Alg. 1, Stage 2;
Sec. 3.4 "Distortion calibration"; Appendix "Reproducibility Checklist":
five bit-widths 2..6).  Appendix "Distortion Model Validation" writes the
same model as alpha * e^{-beta b}; the numbers it prints (beta ~ 3.48 for the
Lloyd-Max curve, Table 6) only agree with the alpha * beta^-b form, which is
the one used here.

Straight-line ordinary least squares, written out.
"""
import numpy as np


def fit_distortion(D, bits):
    """D: [n_comp][n_bits] (or [n_bits]) positive MSE values measured at
    ``bits``.  Returns (alpha, beta, r2) arrays over components.

    slope m and intercept c of  y = ln D  against  x = b;
    alpha = e^c, beta = e^-m, R^2 = 1 - SS_res / SS_tot (1 when SS_tot = 0).
    """
    D = np.atleast_2d(np.asarray(D, dtype=np.float64))
    x = np.asarray(bits, dtype=np.float64)
    if x.size < 2 or D.shape[1] != x.size:
        raise ValueError("need at least two bit-widths, one D per width")
    if np.any(~(D > 0)):
        raise ValueError("distortions must be positive")
    y = np.log(D)
    xm = x.mean()
    ym = y.mean(axis=1, keepdims=True)
    sxx = np.sum((x - xm) ** 2)
    sxy = np.sum((x - xm)[None, :] * (y - ym), axis=1)
    m = sxy / sxx
    c = ym[:, 0] - m * xm
    pred = c[:, None] + m[:, None] * x[None, :]
    ss_res = np.sum((y - pred) ** 2, axis=1)
    ss_tot = np.sum((y - ym) ** 2, axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        r2 = np.where(ss_tot > 0, 1.0 - ss_res / ss_tot, 1.0)
    return np.exp(c), np.exp(-m), r2


def model(alpha, beta, b):
    """D(b) = alpha * beta^-b."""
    return alpha * np.power(beta, -np.asarray(b, dtype=np.float64))
