// The residual-window append shared by the quantize kernels: the tokens of
// an append that stay in the 16-bit window go to their ring slots
// (token t of a (batch entry, kv-head, kind) in slot t mod (R + 32)).
#pragma once
#include "rq_device.h"
#include "rq_internal.h"

namespace rq {

// Rows [t_lo, t_hi) of every (batch entry, kv-head, kind): worker w of n
// (one wave each) copies rows 4 w .. 4 w + 3, then 4 (w + n) .., 16 lanes of
// 16 bytes per 256-byte row.
__device__ __forceinline__ void copy_window(const RingLaunch& r, int worker, int n_workers,
                                            int lane) {
  const int nt = r.t_hi - r.t_lo;
  if (nt <= 0) return;
  const int rows = r.B * r.H * 2 * nt;
  const int cap = r.R + kChunk;
  for (int base = 4 * worker; base < rows; base += 4 * n_workers) {
    const int row = base + (lane >> 4), p = lane & 15;
    if (row < rows) {
      const int t = r.t_lo + row % nt;
      const int z = row / nt, kind = z & 1, bh = z >> 1;   // bh = b H + h
      const uint16_t* src = (kind ? r.v : r.k) + ((size_t)bh * r.n_new + (t - r.n_past)) * kD;
      uint16_t* dst = r.resid + (((size_t)bh * 2 + kind) * cap + (t % cap)) * kD;
      reinterpret_cast<u4*>(dst)[p] = reinterpret_cast<const u4*>(src)[p];
    }
  }
}

}  // namespace rq
