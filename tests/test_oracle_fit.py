"""Pins of the distortion fit (oracle.fit) and of the Lloyd-Max curve."""
import math

import numpy as np
import pytest

import workloads
from oracle import fit, lloydmax
from tests.golden.load import table

T6 = table("table6_lloydmax.txt")


def test_planted_curves_recovered_exactly():
    bits = [1, 2, 3, 4]
    D, a, b = workloads.planted_curves(64, bits, seed=42)
    ah, bh, r2 = fit.fit_distortion(D, bits)
    np.testing.assert_allclose(ah, a, rtol=1e-12)
    np.testing.assert_allclose(bh, b, rtol=1e-12)
    np.testing.assert_allclose(r2, 1.0, atol=1e-12)


@pytest.mark.parametrize("seed", workloads.SEEDS)
def test_planted_curves_with_noise(seed):
    bits = [2, 3, 4, 5, 6]
    D, a, b = workloads.planted_curves(512, bits, seed=seed, noise_sigma=0.02)
    ah, bh, r2 = fit.fit_distortion(D, bits)
    # slope std = sigma / sqrt(sum (b - mean)^2) = 0.02 / sqrt(10)
    assert np.max(np.abs(np.log(bh / b))) < 6 * 0.02 / math.sqrt(10)
    assert np.all(bh > 1) and np.all(r2 > 0.99)


def test_r2_is_squared_correlation():
    # For a one-regressor least-squares line, R^2 equals the squared Pearson
    # correlation of x and y -- an identity independent of the fit code.
    rng = np.random.default_rng(7)
    bits = np.array([2, 3, 4, 5, 6], dtype=float)
    D = np.exp(rng.normal(0, 1, size=(20, 5)) - 1.3 * bits)
    _, _, r2 = fit.fit_distortion(D, bits)
    for i in range(20):
        rho = np.corrcoef(bits, np.log(D[i]))[0, 1]
        assert abs(r2[i] - rho * rho) < 1e-12


def test_fit_of_table6_exact_column():
    # Sec. 3.1: fitting the Lloyd-Max MSE gives alpha ~ 1.36, beta ~ 3.48,
    # R^2 > 0.99 (values read from Table 6, bits 1..6).
    a, b, r2 = fit.fit_distortion(T6[:, 1], T6[:, 0])
    assert round(float(a[0]), 2) == 1.36
    assert round(float(b[0]), 2) == 3.48
    assert r2[0] > 0.99
    # The "Fit" column is the fitted model alpha * beta^-b (within 0.3 %:
    # the table was fitted from unrounded MSE values), and the "Ratio"
    # column is fit / exact.
    np.testing.assert_allclose(fit.model(a[0], b[0], T6[:, 0]), T6[:, 2],
                               rtol=3e-3)
    np.testing.assert_allclose(T6[:, 2] / T6[:, 1], T6[:, 3], atol=6e-4)


def test_fit_rejects_bad_input():
    with pytest.raises(ValueError):
        fit.fit_distortion([1.0], [3])
    with pytest.raises(ValueError):
        fit.fit_distortion([1.0, 0.0], [2, 3])


@pytest.mark.parametrize("b", [1, 2, 3, 4])
def test_lloydmax_mse_matches_table6(b):
    got = lloydmax.mse(lloydmax.centroids(b))
    want = T6[b - 1, 1]
    assert float(f"{got:.3e}") == want


def test_lloydmax_b5_close_to_table6():
    # The printed b=5 value is 0.3 % above the converged optimum (and b=6 is
    # 16 % above; it is not pinned).
    got = lloydmax.mse(lloydmax.centroids(5))
    assert abs(got / T6[4, 1] - 1) < 0.01
    assert got < T6[4, 1]


def test_lloydmax_one_bit_closed_form():
    c = lloydmax.centroids(1)
    np.testing.assert_allclose(c, [-math.sqrt(2 / math.pi),
                                   math.sqrt(2 / math.pi)], rtol=1e-14)
    assert abs(lloydmax.mse(c) - (1 - 2 / math.pi)) < 1e-14


@pytest.mark.parametrize("b", [2, 3, 4])
def test_lloydmax_monte_carlo(b):
    c = lloydmax.centroids(b)
    assert np.allclose(c, -c[::-1])
    x = np.random.default_rng(b).standard_normal(2_000_000)
    idx = np.searchsorted(0.5 * (c[1:] + c[:-1]), x)
    emp = np.mean((x - c[idx]) ** 2)
    assert abs(emp / lloydmax.mse(c) - 1) < 0.01


@pytest.mark.parametrize("b", range(1, 9))
def test_lloydmax_is_a_fixed_point_of_both_conditions(b):
    # Lloyd's conditions define the quantizer: each centroid is the mean of
    # N(0,1) over its cell, measured here by numerical integration on a fine
    # grid (independent of the solver's closed-form cell means), and the
    # centroids are symmetric.
    from scipy import integrate
    c = lloydmax.centroids(b)
    assert np.array_equal(c, -c[::-1])
    t = np.concatenate(([-np.inf], 0.5 * (c[1:] + c[:-1]), [np.inf]))
    for k in range(len(c)):
        lo, hi = max(t[k], -12.0), min(t[k + 1], 12.0)
        pdf = lambda x: np.exp(-0.5 * x * x)
        mass = integrate.quad(pdf, lo, hi, epsabs=0, epsrel=1e-13)[0]
        first = integrate.quad(lambda x: x * pdf(x), lo, hi, epsabs=0,
                               epsrel=1e-13)[0]
        assert abs(first / mass - c[k]) < 1e-9 * max(1.0, abs(c[k]))
