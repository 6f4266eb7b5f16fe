"""Pins of the sensitivity oracle and the host refinements (Alg. 1 Stage 1;
Appendix "Temporal aggregation", "Failure modes", "Distortion Model
Parameters")."""
import numpy as np
import pytest

from oracle import sensitivity as osens


def test_brute_force_loops_tiny():
    rng = np.random.default_rng(0)
    g = rng.standard_normal((2, 3, 5, 128)).astype(np.float32)
    want = []
    for i in range(3):
        acc = 0.0
        for s in range(2):
            seq = 0.0
            for t in range(5):
                seq += sum(float(x) * float(x) for x in g[s, i, t])
            acc += seq / 5
        want.append(acc / 2)
    np.testing.assert_allclose(osens.sensitivity(g), want, rtol=1e-13)


def test_closed_forms():
    # constant gradient c: every position has |g|^2 = 128 c^2
    g = np.full((3, 2, 7, 128), 0.5, dtype=np.float32)
    assert np.allclose(osens.sensitivity(g), 128 * 0.25)
    # one nonzero element at one position of one sequence
    g = np.zeros((4, 2, 8, 128), dtype=np.float32)
    g[1, 1, 3, 17] = 2.0
    np.testing.assert_array_equal(osens.sensitivity(g), [0.0, 4.0 / 8 / 4])


def test_scaling_and_sequence_duplication():
    rng = np.random.default_rng(1)
    g = rng.standard_normal((2, 4, 16, 128)).astype(np.float32)
    w = osens.sensitivity(g)
    # squared norm: doubling the gradients quadruples w
    np.testing.assert_allclose(osens.sensitivity(2 * g), 4 * w, rtol=1e-14)
    # an average over sequences: repeating the set changes nothing
    np.testing.assert_allclose(osens.sensitivity(np.concatenate([g, g])), w,
                               rtol=1e-14)
    # and over positions: repeating every position changes nothing
    np.testing.assert_allclose(osens.sensitivity(np.repeat(g, 3, axis=2)), w,
                               rtol=1e-14)


def test_cap_weights():
    w = np.array([1.0, 2.0, 3.0, 100.0])          # mean 26.5, cap 132.5
    np.testing.assert_array_equal(osens.cap_weights(w), w)
    w = np.array([1.0] * 9 + [91.0])               # mean 10, cap 50
    out = osens.cap_weights(w)
    np.testing.assert_array_equal(out, [1.0] * 9 + [50.0])
    # the ranking of the heads below the cap is kept
    rng = np.random.default_rng(2)
    w = rng.lognormal(0, 2.0, size=200)
    out = osens.cap_weights(w)
    below = w < 5 * w.mean()
    np.testing.assert_array_equal(out[below], w[below])
    assert np.all(out <= 5 * w.mean() * (1 + 1e-15))
    assert np.all(np.argsort(out[below]) == np.argsort(w[below]))


def test_fallback_beta():
    beta = np.array([3.0, 5.0, 6.0, 2.0])          # mean 4
    r2 = np.array([0.99, 0.5, 0.97, 0.2])
    np.testing.assert_array_equal(osens.fallback_beta(beta, r2),
                                  [3.0, 4.0, 6.0, 2.0])
    # every fit good: unchanged
    np.testing.assert_array_equal(osens.fallback_beta(beta, np.ones(4)), beta)


@pytest.mark.parametrize("S,n,T", [(1, 1, 1), (3, 5, 96)])
def test_shapes(S, n, T):
    g = np.ones((S, n, T, 128), dtype=np.float32)
    assert osens.sensitivity(g).shape == (n,)
