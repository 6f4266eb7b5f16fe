"""Bit allocation (oracle).

Problem (Sec. 3.1, eq. 1, generalised to per-component (alpha_i, beta_i) as
in Sec. 3.4 "K/V separation" and Alg. 2):

    minimise  J(b) = sum_i w_i * alpha_i * beta_i^-b_i
    s.t.      sum_i b_i = B,   bmin <= b_i <= bmax,

with B = round(avg_bits * n) (Sec. 3.1 writes B as the rounded product of
the average bit-width and the component count).

* ``waterfill``: the continuous optimum.  Its plain definition is the KKT
  point of the convex problem (Appendix "Proof of Theorem 1"): every free
  component satisfies w_i alpha_i ln(beta_i) beta_i^-b_i = lambda, and the
  bounded ones sit at a bound.  Written as b_i(nu) =
  clip((ln(w_i alpha_i ln beta_i) - nu) / ln beta_i, bmin, bmax) with
  nu = ln lambda chosen so that sum_i b_i(nu) = B (found by bisection, then
  solved exactly on the resulting free set).
* ``waterfill_iterative``: the paper's own bound-handling loop (Appendix
  "Proof of Theorem 1", "Iterative waterfilling"): solve with all free, clip
  violators to their bound and fix them, update the budget, repeat.
* ``greedy``: the integer allocation of Stage 3 of Alg. 1 / Alg. 2, written
  from its definition rather than its listing.  Raising component i from b
  to b+1 lowers J by the marginal gain w_i [D_i(b) - D_i(b+1)]
  = w_i alpha_i beta_i^-b (1 - 1/beta_i) (Sec. 3.3; Proposition 3), a
  strictly decreasing function of b when beta_i > 1.  Starting every
  component at bmin, the greedy rule spends the remaining R = B - n*bmin
  bits on the R largest gains; because each component's gains fall with b,
  that is the same as ranking all n (bmax - bmin) increments (i, b) at once
  and keeping the top R.  Gains are compared through their logarithm,
  evaluated in IEEE double as log(w) + log(alpha) - b*log(beta) +
  log1p(-1/beta) (left to right); equal keys go to the lower index, then the
  lower b (the paper does not say).
* ``brute_force``: exhaustive search of the integer problem (tiny n).
"""
import itertools
import math

import numpy as np


class Infeasible(ValueError):
    pass


def budget(n, avg_bits):
    """B = round(avg_bits * n), halves away from zero (llround)."""
    x = avg_bits * n
    return int(math.floor(x + 0.5)) if x >= 0 else -int(math.floor(-x + 0.5))


def J(w, alpha, beta, b):
    w, alpha, beta, b = (np.asarray(a, dtype=np.float64)
                         for a in (w, alpha, beta, b))
    return float(np.sum(w * alpha * beta ** (-b)))


def _check(w, alpha, beta, B, bmin, bmax):
    w, alpha, beta = (np.asarray(a, dtype=np.float64) for a in (w, alpha, beta))
    n = w.size
    if not (alpha.size == n and beta.size == n):
        raise ValueError("w, alpha, beta must have the same length")
    if np.any(~(w > 0)) or np.any(~(alpha > 0)) or np.any(~(beta > 1)):
        raise ValueError("need w > 0, alpha > 0, beta > 1")
    if bmin > bmax:
        raise ValueError("bmin > bmax")
    if not (n * bmin <= B <= n * bmax):
        raise Infeasible(f"budget {B} outside [{n * bmin}, {n * bmax}]")
    return w, alpha, beta


def waterfill(w, alpha, beta, B, bmin, bmax):
    """Continuous optimum b* (float64 array)."""
    w, alpha, beta = _check(w, alpha, beta, B, bmin, bmax)
    ell = np.log(beta)
    k = np.log(w * alpha * ell)

    def bits_at(nu):
        return np.clip((k - nu) / ell, bmin, bmax)

    # S(nu) = sum b_i(nu) is continuous and non-increasing in nu.
    lo = float(np.min(k - bmax * ell)) - 1.0     # every b_i = bmax
    hi = float(np.max(k - bmin * ell)) + 1.0     # every b_i = bmin
    for _ in range(400):
        mid = 0.5 * (lo + hi)
        if np.sum(bits_at(mid)) > B:
            lo = mid
        else:
            hi = mid
    b = bits_at(0.5 * (lo + hi))
    free = (b > bmin) & (b < bmax)
    if np.any(free):
        fixed_sum = float(np.sum(b[~free]))
        nu = (np.sum(k[free] / ell[free]) - (B - fixed_sum)) / np.sum(
            1.0 / ell[free])
        b = b.copy()
        b[free] = (k[free] - nu) / ell[free]
    return b


def waterfill_iterative(w, alpha, beta, B, bmin, bmax, max_rounds=None):
    """The paper's clip-fix-repeat loop, kept as written."""
    w, alpha, beta = _check(w, alpha, beta, B, bmin, bmax)
    n = w.size
    ell = np.log(beta)
    k = np.log(w * alpha * ell)
    b = np.zeros(n)
    free = np.ones(n, dtype=bool)
    budget_left = float(B)
    for _ in range(max_rounds or n):
        nu = (np.sum(k[free] / ell[free]) - budget_left) / np.sum(
            1.0 / ell[free])
        b[free] = (k[free] - nu) / ell[free]
        low = free & (b < bmin)
        high = free & (b > bmax)
        if not (np.any(low) or np.any(high)):
            break
        b[low] = bmin
        b[high] = bmax
        free &= ~(low | high)
        budget_left = B - float(np.sum(b[~free]))
        if not np.any(free):
            break
    return b


def gain_key(w, alpha, beta, b):
    """log of w * alpha * beta^-b * (1 - 1/beta), left to right."""
    return (math.log(w) + math.log(alpha) - float(b) * math.log(beta)
            + math.log1p(-1.0 / beta))


def greedy(w, alpha, beta, B, bmin, bmax):
    """Integer allocation (Alg. 1 Stage 3 / Alg. 2; Proposition 3): every
    component at bmin plus one bit for each of the R = B - n*bmin largest
    marginal gains among all increments (i, b), bmin <= b < bmax.  Returns
    an int32 array."""
    w, alpha, beta = _check(w, alpha, beta, B, bmin, bmax)
    n = w.size
    R = B - n * bmin
    steps = sorted((-gain_key(w[i], alpha[i], beta[i], b), i, b)
                   for i in range(n) for b in range(bmin, bmax))
    bits = np.full(n, bmin, dtype=np.int64)
    for _, i, _ in steps[:R]:
        bits[i] += 1
    return bits.astype(np.int32)


def brute_force(w, alpha, beta, B, bmin, bmax):
    """Exhaustive minimiser of J over integer vectors (small n only).
    Returns (best_J, list of all minimising vectors)."""
    w, alpha, beta = _check(w, alpha, beta, B, bmin, bmax)
    n = w.size
    best, arg = math.inf, []
    for cand in itertools.product(range(bmin, bmax + 1), repeat=n):
        if sum(cand) != B:
            continue
        j = J(w, alpha, beta, cand)
        if j < best * (1 - 1e-13):
            best, arg = j, [cand]
        elif j <= best * (1 + 1e-13):
            arg.append(cand)
    return best, arg


def theorem1(w, beta, avg_bits):
    """Closed form of Theorem 1 (eq. 2): shared beta, no active bound."""
    lw = np.log(np.asarray(w, dtype=np.float64))
    return avg_bits + (lw - lw.mean()) / math.log(beta)
