"""Lloyd-Max scalar quantizer of the standard normal (oracle).

The TurboQuant-style base quantizer maps each rotated coordinate to one of
2^b centroids of the Lloyd-Max quantizer of the coordinate distribution; the
paper's Table 6 (Appendix "Distortion Model Validation") lists the exact MSE
of that quantizer for unit-variance Gaussian data, b = 1..6.

Lloyd's two conditions, iterated to a fixed point in fp64:
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


def centroids(b, iters=100000, tol=1e-15):
    """2^b Lloyd-Max centroids of N(0,1), ascending (float64)."""
    L = 1 << b
    # start from equal-probability cell means
    c = np.sort(np.array([0.0]) if L == 1 else
                np.linspace(-1.0, 1.0, L) * (1.0 + 0.5 * b))
    for _ in range(iters):
        e = _cells(c)
        pa, pb = _phi(e[:-1]), _phi(e[1:])
        pa[0] = 0.0
        pb[-1] = 0.0
        mass = ndtr(e[1:]) - ndtr(e[:-1])
        cn = (pa - pb) / mass
        # exact symmetry of the standard normal: c_k = -c_{L-1-k}
        cn = 0.5 * (cn - cn[::-1])
        if np.max(np.abs(cn - c)) <= tol:
            c = cn
            break
        c = cn
    return c


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
