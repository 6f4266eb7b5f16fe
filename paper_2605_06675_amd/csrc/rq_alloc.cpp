// Host-side distortion fit and bit allocation.
//
// Fit (Alg. 1 Stage 2): ordinary least squares of ln D against b, giving
// ln alpha (intercept) and -ln beta (slope).
//
// Allocation (eq. 1 with per-component alpha_i, beta_i; Theorem 1 and its
// bound handling; Alg. 1 Stage 3 / Alg. 2):
//  * continuous optimum: with l_i = ln beta_i and k_i = ln(w_i alpha_i l_i),
//    the KKT point is b_i(nu) = clamp((k_i - nu) / l_i, bmin, bmax) with
//    sum_i b_i(nu) = B.  S(nu) = sum_i b_i(nu) is piecewise linear and
//    non-increasing with breakpoints k_i - bmax l_i (leaves bmax) and
//    k_i - bmin l_i (reaches bmin); a sweep over the sorted breakpoints
//    finds the segment holding B and solves it in closed form;
//  * integer optimum: a max-heap of marginal gains, one bit at a time.
#include <algorithm>
#include <cmath>
#include <queue>
#include <vector>

#include "rq_host.h"

namespace rq {

rq_status fit_distortion(const double* mse, int n_comp, const int32_t* bits,
                         int n_bits, double* alpha, double* beta, double* r2) {
  double xm = 0;
  for (int j = 0; j < n_bits; ++j) xm += bits[j];
  xm /= n_bits;
  double sxx = 0;
  for (int j = 0; j < n_bits; ++j) sxx += (bits[j] - xm) * (bits[j] - xm);
  std::vector<double> y(n_bits);
  for (int i = 0; i < n_comp; ++i) {
    double ym = 0;
    for (int j = 0; j < n_bits; ++j) {
      y[j] = std::log(mse[(size_t)i * n_bits + j]);
      ym += y[j];
    }
    ym /= n_bits;
    double sxy = 0;
    for (int j = 0; j < n_bits; ++j) sxy += (bits[j] - xm) * (y[j] - ym);
    const double slope = sxy / sxx;
    const double icept = ym - slope * xm;
    double ss_res = 0, ss_tot = 0;
    for (int j = 0; j < n_bits; ++j) {
      const double e = y[j] - (icept + slope * bits[j]);
      ss_res += e * e;
      ss_tot += (y[j] - ym) * (y[j] - ym);
    }
    if (alpha) alpha[i] = std::exp(icept);
    if (beta) beta[i] = std::exp(-slope);
    if (r2) r2[i] = ss_tot > 0 ? 1.0 - ss_res / ss_tot : 1.0;
  }
  return RQ_OK;
}

int64_t budget(int n, double avg_bits) { return std::llround(avg_bits * n); }

void waterfill(int n, const double* w, const double* alpha, const double* beta,
               int64_t B, int bmin, int bmax, double* out) {
  std::vector<double> l(n), k(n);
  for (int i = 0; i < n; ++i) {
    l[i] = std::log(beta[i]);
    k[i] = std::log(w[i] * alpha[i] * l[i]);
  }
  if (B >= (int64_t)n * bmax || bmin == bmax) {
    for (int i = 0; i < n; ++i) out[i] = B >= (int64_t)n * bmax ? bmax : bmin;
    return;
  }
  if (B <= (int64_t)n * bmin) {
    for (int i = 0; i < n; ++i) out[i] = bmin;
    return;
  }
  struct Ev {
    double nu;
    int i;
    bool upper;  // true: i leaves bmax here; false: i reaches bmin here
  };
  std::vector<Ev> ev;
  ev.reserve(2 * (size_t)n);
  for (int i = 0; i < n; ++i) {
    ev.push_back({k[i] - bmax * l[i], i, true});
    ev.push_back({k[i] - bmin * l[i], i, false});
  }
  std::sort(ev.begin(), ev.end(), [](const Ev& a, const Ev& b) {
    if (a.nu != b.nu) return a.nu < b.nu;
    return a.upper && !b.upper;
  });
  // state left of the first breakpoint: everything at bmax
  double fixed = (double)n * bmax, A = 0, C = 0;
  double nu_prev = -INFINITY;
  double nu_sol = ev.back().nu;
  for (size_t e = 0; e < ev.size(); ++e) {
    const double nu = ev[e].nu;
    const double S = fixed + A - nu * C;  // S at this breakpoint
    if (S <= (double)B) {
      // the solution lies in [nu_prev, nu]
      nu_sol = C > 0 ? (fixed + A - (double)B) / C : nu;
      if (nu_sol < nu_prev) nu_sol = nu_prev;
      if (nu_sol > nu) nu_sol = nu;
      break;
    }
    const int i = ev[e].i;
    if (ev[e].upper) {
      fixed -= bmax;
      A += k[i] / l[i];
      C += 1.0 / l[i];
    } else {
      fixed += bmin;
      A -= k[i] / l[i];
      C -= 1.0 / l[i];
    }
    nu_prev = nu;
  }
  // exact solve on the free set of that segment (sums recomputed directly)
  double f2 = 0, A2 = 0, C2 = 0;
  std::vector<char> fr(n);
  for (int i = 0; i < n; ++i) {
    const double bi = (k[i] - nu_sol) / l[i];
    if (bi >= bmax) {
      f2 += bmax;
    } else if (bi <= bmin) {
      f2 += bmin;
    } else {
      fr[i] = 1;
      A2 += k[i] / l[i];
      C2 += 1.0 / l[i];
    }
  }
  if (C2 > 0) nu_sol = (f2 + A2 - (double)B) / C2;
  for (int i = 0; i < n; ++i) {
    double bi = (k[i] - nu_sol) / l[i];
    out[i] = bi < bmin ? bmin : (bi > bmax ? bmax : bi);
  }
}

static inline double gain_key(double w, double a, double be, int b) {
  return std::log(w) + std::log(a) - (double)b * std::log(be) +
         std::log1p(-1.0 / be);
}

void greedy(int n, const double* w, const double* alpha, const double* beta,
            int64_t B, int bmin, int bmax, int32_t* out) {
  struct Item {
    double key;
    int i;
  };
  // top = largest key; equal keys: lowest index first
  auto lower = [](const Item& a, const Item& b) {
    return a.key < b.key || (a.key == b.key && a.i > b.i);
  };
  std::priority_queue<Item, std::vector<Item>, decltype(lower)> heap(lower);
  for (int i = 0; i < n; ++i) {
    out[i] = bmin;
    if (bmin < bmax) heap.push({gain_key(w[i], alpha[i], beta[i], bmin), i});
  }
  for (int64_t R = B - (int64_t)n * bmin; R > 0; --R) {
    const Item top = heap.top();
    heap.pop();
    const int i = top.i;
    out[i] += 1;
    if (out[i] < bmax) heap.push({gain_key(w[i], alpha[i], beta[i], out[i]), i});
  }
}

}  // namespace rq
