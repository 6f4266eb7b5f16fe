"""Pins of the allocation oracle (oracle.alloc) against what the paper and
the mathematics fix."""
import math

import numpy as np
import pytest

import workloads
from oracle import alloc


def _rand_instance(rng, n, shared=False):
    w = rng.lognormal(0, 0.8, n)
    if shared:
        a = np.full(n, rng.uniform(0.1, 5))
        b = np.full(n, rng.uniform(3.6, 5.3))
    else:
        a = rng.lognormal(0, 1, n)
        b = rng.uniform(2.0, 6.0, n)
    return w, a, b


def test_theorem1_closed_form():
    # Shared alpha, beta and no active bound: b_i = avg + (ln w_i - mean) /
    # ln beta (Theorem 1, eq. 2).
    rng = np.random.default_rng(1)
    n, beta, avg = 64, 3.48, 4.0
    w = rng.lognormal(0, 0.3, n)
    B = alloc.budget(n, avg)
    b = alloc.waterfill(w, np.full(n, 1.36), np.full(n, beta), B, 0, 20)
    np.testing.assert_allclose(b, alloc.theorem1(w, beta, avg), atol=1e-10)
    assert abs(b.sum() - B) < 1e-10 * B


@pytest.mark.parametrize("seed", workloads.SEEDS)
def test_waterfill_budget_and_kkt(seed):
    # Sum b = B exactly, and the KKT conditions of eq. 1: the marginal
    # w alpha ln(beta) beta^-b is equal (lambda) on free components, at most
    # lambda at bmin and at least lambda at bmax.
    rng = np.random.default_rng(seed)
    w, a, b = _rand_instance(rng, 300)
    B = alloc.budget(300, 3.0)
    x = alloc.waterfill(w, a, b, B, 2, 5)
    assert abs(x.sum() - B) < 1e-9
    marg = w * a * np.log(b) * b ** (-x)
    free = (x > 2 + 1e-9) & (x < 5 - 1e-9)
    lam = np.median(marg[free])
    np.testing.assert_allclose(marg[free], lam, rtol=1e-8)
    assert np.all(marg[x <= 2 + 1e-9] <= lam * (1 + 1e-8))
    assert np.all(marg[x >= 5 - 1e-9] >= lam * (1 - 1e-8))


def test_gain_ratio_is_am_over_gm():
    # Theorem 2: J_uniform / J_opt = AM(w) / GM(w) with no active bounds.
    rng = np.random.default_rng(3)
    n, alpha, beta, avg = 512, 1.5, 4.2, 4.0
    w = rng.lognormal(0, 0.5, n)
    B = alloc.budget(n, avg)
    bs = alloc.waterfill(w, np.full(n, alpha), np.full(n, beta), B, -50, 50)
    ju = alloc.J(w, np.full(n, alpha), np.full(n, beta), np.full(n, avg))
    jo = alloc.J(w, np.full(n, alpha), np.full(n, beta), bs)
    am, gm = w.mean(), math.exp(np.log(w).mean())
    assert abs(ju / jo - am / gm) < 1e-12 * am / gm


def test_corollary1_lognormal_gain():
    # Corollary 1: ln w ~ N(mu, s^2) gives J_u / J* -> exp(s^2 / 2).
    rng = np.random.default_rng(4)
    for s in (0.5, 0.76):
        w = rng.lognormal(0.3, s, 200_000)
        ratio = w.mean() / math.exp(np.log(w).mean())
        assert abs(ratio / math.exp(s * s / 2) - 1) < 0.01


def test_two_head_offsets():
    # Sec. 3.1: a head e times more sensitive gets 1/ln(beta) more bits
    # (0.80 at beta = 3.48); Sec. 3.4: a 2x sensitivity error moves the
    # allocation by ln 2 / ln beta (0.43 at beta = 5).
    for beta, ratio, want in ((3.48, math.e, 0.80), (5.0, 2.0, 0.43)):
        b = alloc.waterfill([1.0, ratio], [1.0, 1.0], [beta, beta], 8, 0, 8)
        assert round(b[1] - b[0], 2) == want
        assert abs((b[1] - b[0]) - math.log(ratio) / math.log(beta)) < 1e-12


def test_iterative_waterfilling_matches_kkt_one_sided():
    # The paper's clip-and-fix loop reaches the KKT point when only the
    # upper bound binds.
    rng = np.random.default_rng(5)
    w = rng.lognormal(0, 1.5, 200)
    a, b = np.ones(200), np.full(200, 4.0)
    B = alloc.budget(200, 3.0)
    x1 = alloc.waterfill(w, a, b, B, -100, 4.5)
    x2 = alloc.waterfill_iterative(w, a, b, B, -100, 4.5)
    assert np.any(x1 >= 4.5 - 1e-9)
    np.testing.assert_allclose(x1, x2, atol=1e-9)


@pytest.mark.parametrize("seed", range(6))
def test_greedy_equals_brute_force(seed):
    # Proposition 3: with convex D the greedy allocation is optimal.
    rng = np.random.default_rng(100 + seed)
    for _ in range(40):
        n = int(rng.integers(2, 6))
        bmin = int(rng.integers(1, 3))
        bmax = bmin + int(rng.integers(1, 4))
        B = int(rng.integers(n * bmin, n * bmax + 1))
        w, a, b = _rand_instance(rng, n)
        g = alloc.greedy(w, a, b, B, bmin, bmax)
        best, args = alloc.brute_force(w, a, b, B, bmin, bmax)
        assert g.sum() == B
        assert abs(alloc.J(w, a, b, g) - best) <= 1e-12 * best
        assert tuple(int(v) for v in g) in args


def test_uniform_special_case():
    # All components identical: the bits are as equal as possible; the
    # extra bits go to the lowest indices (ties broken by index).
    n, avg = 10, 2.3
    B = alloc.budget(n, avg)
    g = alloc.greedy(np.ones(n), np.ones(n), np.full(n, 4.0), B, 1, 8)
    assert list(g) == [3, 3, 3, 2, 2, 2, 2, 2, 2, 2]


def test_qwen3_8b_remaining_budget():
    # Sec. 3.3 / Alg. 2: Qwen3-8B has N = 288 heads (576 components); at
    # avg 4 bits and bmin = 2, R = B - 2N*bmin = 1152.
    n = 2 * 36 * 8
    B = alloc.budget(n, 4.0)
    assert B - n * 2 == 1152


@pytest.mark.parametrize("name", ["llama3-8b-kv-b16-t8192-kivi-2.5b",
                                  "qwen3-8b-kv-b8-t32768-quarot-4b",
                                  "llama3-70b-kv-b4-t32768-turbo-3b",
                                  "qwen3-32b-kv-b1-t131072-kivi-2b"])
def test_workload_allocations(name):
    wl = workloads.WORKLOADS[name]
    w, a, b = workloads.allocation_inputs(wl)
    n = wl.n_comp
    B = alloc.budget(n, wl.avg_bits)
    lo, hi = min(wl.bit_set), max(wl.bit_set)
    g = alloc.greedy(w, a, b, B, lo, hi)
    c = alloc.waterfill(w, a, b, B, lo, hi)
    assert g.sum() == B and g.min() >= lo and g.max() <= hi
    assert abs(c.sum() - B) < 1e-9 * B
    # integer and continuous optima stay within one bit of each other, and
    # the integer optimum is never better than the continuous one
    assert np.max(np.abs(g - c)) < 1.0
    assert alloc.J(w, a, b, g) >= alloc.J(w, a, b, c) * (1 - 1e-12)


def test_infeasible_budget():
    with pytest.raises(alloc.Infeasible):
        alloc.greedy([1, 1], [1, 1], [4, 4], 9, 2, 4)
    with pytest.raises(alloc.Infeasible):
        alloc.waterfill([1, 1], [1, 1], [4, 4], 3, 2, 4)
    with pytest.raises(ValueError):
        alloc.greedy([1, -1], [1, 1], [4, 4], 6, 2, 4)
