"""Lloyd-Max scalar quantizer of the standard normal (oracle).

The TurboQuant-style base quantizer maps each rotated coordinate to one of
2^b centroids of the Lloyd-Max quantizer of the coordinate distribution; the
paper's Table 6 (Appendix "Distortion Model Validation") lists the exact MSE
of that quantizer for unit-variance Gaussian data, b = 1..6.

Lloyd's two conditions, solved for their fixed point in fp64:
  thresholds are midpoints of adjacent centroids;
  each centroid is the conditional mean of N(0,1) on its cell,
      c_k = (phi(t_{k-1}) - phi(t_k)) / (Phi(t_k) - Phi(t_{k-1})).
"""
import math

import numpy as np
from scipy.special import ndtr


def _phi(x):
    return np.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)


def _cells(c):
    t = 0.5 * (c[1:] + c[:-1])
    return np.concatenate(([-np.inf], t, [np.inf]))


def _upper_cells(u):
    """Cells [a_k, b_k) of the upper-half centroids u (ascending, > 0): the
    first starts at the symmetric midpoint 0, the last runs to infinity."""
    mid = 0.5 * (u[1:] + u[:-1])
    return np.concatenate(([0.0], mid)), np.concatenate((mid, [np.inf]))


def _cell_means(a, b):
    """Mean of N(0,1) on [a, b), 0 <= a < b, with its partial derivatives in
    a and b.  Upper-tail probabilities avoid cancellation far out."""
    pa, pb = _phi(a), np.where(np.isinf(b), 0.0, _phi(b))
    mass = ndtr(-a) - ndtr(-b)
    m = (pa - pb) / mass
    dm_da = pa * (m - a) / mass
    dm_db = np.where(np.isinf(b), 0.0, pb * (np.where(np.isinf(b), 0.0, b) - m) / mass)
    return m, dm_da, dm_db


def centroids(b, lloyd_iters=2000):
    """2^b Lloyd-Max centroids of N(0,1), ascending (float64).

    N(0,1) is symmetric, so the levels are +-u with u the upper half and the
    middle threshold at 0.  Plain Lloyd iterations bring u near the fixed
    point; they contract slowly at many levels, so Newton steps on the
    fixed-point equations u_k = E[X | X in cell k] (a tridiagonal system,
    since cell k's ends are the midpoints with u_{k-1} and u_{k+1}) finish
    the solve to rounding level."""
    L = 1 << b
    h = L // 2
    u = (np.arange(h) + 0.5) * (3.0 + 0.5 * b) / h
    for _ in range(lloyd_iters):
        u = _cell_means(*_upper_cells(u))[0]
    for _ in range(100):
        a, e = _upper_cells(u)
        m, dm_da, dm_db = _cell_means(a, e)
        F = u - m
        # d m_k / d u_j: the lower end a_k = (u_{k-1} + u_k) / 2 for k >= 1,
        # the upper end b_k = (u_k + u_{k+1}) / 2 for k < h - 1
        J = np.eye(h)
        for k in range(h):
            if k >= 1:
                J[k, k - 1] -= 0.5 * dm_da[k]
                J[k, k] -= 0.5 * dm_da[k]
            if k < h - 1:
                J[k, k] -= 0.5 * dm_db[k]
                J[k, k + 1] -= 0.5 * dm_db[k]
        step = np.linalg.solve(J, F)
        u = u - step
        if np.max(np.abs(step)) <= 1e-16:
            break
    return np.concatenate((-u[::-1], u))


def mse(c):
    """E[(X - Q(X))^2] for X ~ N(0,1) and nearest-centroid Q."""
    e = _cells(np.asarray(c, dtype=np.float64))
    a, b = e[:-1], e[1:]
    pa, pb = _phi(a), _phi(b)
    fa, fb = np.where(np.isinf(a), 0.0, a), np.where(np.isinf(b), 0.0, b)
    apa, bpb = fa * pa, fb * pb        # x phi(x) -> 0 at +-infinity
    mass = ndtr(b) - ndtr(a)
    second = mass + apa - bpb          # integral of x^2 phi over the cell
    first = pa - pb                    # integral of x phi over the cell
    return float(np.sum(second - 2.0 * c * first + c * c * mass))


def thresholds_f32(c):
    """Decision thresholds as fp32: midpoints computed in fp64, rounded."""
    c = np.asarray(c, dtype=np.float64)
    return (0.5 * (c[1:] + c[:-1])).astype(np.float32)
