// Lloyd-Max quantizer of the standard normal distribution: the per-
// coordinate codebook of the TurboQuant-style quantizer (Sec. 2; Sec. 3.1,
// whose Table 6 lists its MSE for b = 1..6).  Host only.
//
// Lloyd's two optimality conditions are solved for their fixed point in
// double precision: the decision thresholds are the midpoints of adjacent
// centroids, and each centroid is the mean of N(0,1) restricted to its cell,
//   c_k = (phi(t_{k-1}) - phi(t_k)) / (Phi(t_k) - Phi(t_{k-1})).
// The distribution is symmetric, so only the upper half of the levels is
// solved; the lower half mirrors it.
#include <cmath>
#include <cstring>
#include <mutex>
#include <vector>

#include "rq_host.h"
#include "rq_internal.h"

namespace {

const double kInvSqrt2Pi = 0.3989422804014327;
const double kInvSqrt2 = 0.7071067811865476;

double phi(double x) { return std::isinf(x) ? 0.0 : kInvSqrt2Pi * std::exp(-0.5 * x * x); }

// Mean of N(0,1) on [a, b), 0 <= a < b <= inf, and its derivatives in the
// two ends.  Upper-tail masses (erfc) keep far cells accurate.
struct CellMean {
  double m, d_lo, d_hi;
};

CellMean cell_mean(double a, double b) {
  const double pa = phi(a), pb = phi(b);
  const double qa = 0.5 * std::erfc(a * kInvSqrt2);
  const double qb = std::isinf(b) ? 0.0 : 0.5 * std::erfc(b * kInvSqrt2);
  const double mass = qa - qb;
  CellMean r;
  r.m = (pa - pb) / mass;
  r.d_lo = pa * (r.m - a) / mass;
  r.d_hi = std::isinf(b) ? 0.0 : pb * (b - r.m) / mass;
  return r;
}

// Centroids of the 2^b-level quantizer, ascending.  The upper half u is
// solved; the lower half is its mirror image and the middle threshold 0.
// Lloyd iterations approach the fixed point; Newton steps on the fixed-point
// equations u_k = mean of cell k finish it (the Jacobian is tridiagonal:
// cell k is bounded by the midpoints with its two neighbours).
std::vector<double> lloyd_max(int b) {
  const int L = 1 << b, h = L / 2;
  std::vector<double> u(h), lo(h), hi(h);
  auto cells = [&] {
    for (int k = 0; k < h; ++k) {
      lo[k] = k == 0 ? 0.0 : 0.5 * (u[k - 1] + u[k]);
      hi[k] = k == h - 1 ? INFINITY : 0.5 * (u[k] + u[k + 1]);
    }
  };
  for (int k = 0; k < h; ++k) u[k] = (k + 0.5) * (3.0 + 0.5 * b) / h;
  for (int it = 0; it < 3000; ++it) {
    cells();
    for (int k = 0; k < h; ++k) u[k] = cell_mean(lo[k], hi[k]).m;
  }
  std::vector<double> sub(h), diag(h), sup(h), rhs(h);
  for (int it = 0; it < 100; ++it) {
    cells();
    for (int k = 0; k < h; ++k) {
      const CellMean c = cell_mean(lo[k], hi[k]);
      rhs[k] = u[k] - c.m;
      sub[k] = k > 0 ? -0.5 * c.d_lo : 0.0;
      sup[k] = k < h - 1 ? -0.5 * c.d_hi : 0.0;
      diag[k] = 1.0 + (k > 0 ? -0.5 * c.d_lo : 0.0) + (k < h - 1 ? -0.5 * c.d_hi : 0.0);
    }
    // tridiagonal elimination, then back substitution
    for (int k = 1; k < h; ++k) {
      const double f = sub[k] / diag[k - 1];
      diag[k] -= f * sup[k - 1];
      rhs[k] -= f * rhs[k - 1];
    }
    double big = 0.0;
    for (int k = h - 1; k >= 0; --k) {
      const double x = (rhs[k] - (k < h - 1 ? sup[k] * rhs[k + 1] : 0.0)) / diag[k];
      rhs[k] = x;
    }
    for (int k = 0; k < h; ++k) {
      u[k] -= rhs[k];
      big = std::fmax(big, std::fabs(rhs[k]));
    }
    if (big <= 1e-16) break;
  }
  std::vector<double> c(L);
  for (int k = 0; k < h; ++k) {
    c[h + k] = u[k];
    c[h - 1 - k] = -u[k];
  }
  return c;
}

}  // namespace

namespace rq {

const float* turbo_table() {
  static std::vector<float> table;
  static std::once_flag once;
  std::call_once(once, [] {
    table.assign(RQ_TURBO_TABLE_FLOATS, 0.0f);
    for (int b = 1; b <= 8; ++b) {
      const std::vector<double> c = lloyd_max(b);
      const int L = 1 << b;
      float* th = table.data() + (b - 1) * 512;
      float* ce = th + 256;
      for (int k = 0; k < 256; ++k) th[k] = INFINITY;
      for (int k = 0; k + 1 < L; ++k) th[k] = (float)(0.5 * (c[k] + c[k + 1]));
      for (int k = 0; k < L; ++k) ce[k] = (float)c[k];
    }
  });
  return table.data();
}

}  // namespace rq
