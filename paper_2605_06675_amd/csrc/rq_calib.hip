// Distortion sweep: for every component and bit-width, quantize and
// dequantize the calibration vectors and sum the squared error.  One wave
// per (component, 32-token block) reads its block once and runs every
// bit-width from registers; per-block sums (fp64) are reduced in a fixed
// order by a second kernel, so results do not depend on scheduling.
#include "rq_device.h"
#include "rq_internal.h"

namespace rq {

namespace {

constexpr int kWave = 64;

__device__ __forceinline__ double wave_sum(double v) {
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, kWave);
  return v;
}

__device__ __forceinline__ float dpp_xor1(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF,
                                      0xF, true));
}

// error of one element: x - (u*s + z) = (x - z) - u*s, one rounding after
// the exact product
__device__ __forceinline__ double sq_err(float d, int u, float sf) {
  const float e = __builtin_fmaf(-(float)u, sf, d);
  return (double)e * (double)e;
}

__global__ void __launch_bounds__(kWave)
calib_kernel(CalibLaunch a) {
  const int blk = blockIdx.x, comp = blockIdx.y, lane = threadIdx.x;
  const int n_blk = a.T / kChunk;
  const uint16_t* x = a.x + ((size_t)comp * a.T + (size_t)blk * kChunk) * kD;
  double* part = a.partial + ((size_t)comp * n_blk + blk) * a.n_bits;

  if (a.family == RQ_KIVI && !a.is_value) {
    // keys: channels 2l, 2l+1 across the 32 tokens
    float x0[kChunk], x1[kChunk];
    float mn0 = INFINITY, mx0 = -INFINITY, mn1 = INFINITY, mx1 = -INFINITY;
#pragma unroll
    for (int t = 0; t < kChunk; ++t) {
      const uint32_t w = *reinterpret_cast<const uint32_t*>(x + t * kD + 2 * lane);
      x0[t] = widen(w & 0xffffu, a.is_bf16);
      x1[t] = widen(w >> 16, a.is_bf16);
      mn0 = __builtin_fminf(mn0, x0[t]);
      mx0 = __builtin_fmaxf(mx0, x0[t]);
      mn1 = __builtin_fminf(mn1, x1[t]);
      mx1 = __builtin_fmaxf(mx1, x1[t]);
    }
    for (int j = 0; j < a.n_bits; ++j) {
      const float qmax = (float)((1 << a.bits[j]) - 1);
      const AsymParams p0 = asym_params(mn0, mx0, qmax);
      const AsymParams p1 = asym_params(mn1, mx1, qmax);
      const float s0 = f16_to_f32(p0.s16), s1 = f16_to_f32(p1.s16);
      double acc = 0.0;
#pragma unroll
      for (int t = 0; t < kChunk; ++t) {
        acc += sq_err(x0[t] - p0.zf, asym_code(x0[t], p0, qmax), s0);
        acc += sq_err(x1[t] - p1.zf, asym_code(x1[t], p1, qmax), s1);
      }
      acc = wave_sum(acc);
      if (lane == 0) part[j] = acc;
    }
    return;
  }

  if (a.family == RQ_KIVI) {
    // values: token l/2, channel groups 2*(l&1) and 2*(l&1)+1
    const int t = lane >> 1, half = lane & 1;
    float xv[64];
    const uint4* s4 = reinterpret_cast<const uint4*>(x + t * kD + half * 64);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint4 w = s4[i];
      const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        xv[8 * i + 2 * e] = widen(ww[e] & 0xffffu, a.is_bf16);
        xv[8 * i + 2 * e + 1] = widen(ww[e] >> 16, a.is_bf16);
      }
    }
    float mn[2], mx[2];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      mn[g] = xv[32 * g];
      mx[g] = xv[32 * g];
#pragma unroll
      for (int i = 1; i < 32; ++i) {
        mn[g] = __builtin_fminf(mn[g], xv[32 * g + i]);
        mx[g] = __builtin_fmaxf(mx[g], xv[32 * g + i]);
      }
    }
    for (int j = 0; j < a.n_bits; ++j) {
      const float qmax = (float)((1 << a.bits[j]) - 1);
      double acc = 0.0;
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const AsymParams p = asym_params(mn[g], mx[g], qmax);
        const float sf = f16_to_f32(p.s16);
#pragma unroll
        for (int i = 0; i < 32; ++i) {
          const float v = xv[32 * g + i];
          acc += sq_err(v - p.zf, asym_code(v, p, qmax), sf);
        }
      }
      acc = wave_sum(acc);
      if (lane == 0) part[j] = acc;
    }
    return;
  }

  // QuaRot: rotate each token (same butterflies as the quantizer), then
  // measure the error of the symmetric levels in the rotated domain, which
  // equals the original-domain error up to fp32 rounding (the rotation is
  // orthonormal).
  const int t = lane >> 1, hb = lane & 1;
  float v[64];
#pragma unroll
  for (int part2 = 0; part2 < 2; ++part2) {
    const uint4* s4 = reinterpret_cast<const uint4*>(x + t * kD + part2 * 64 + hb * 32);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint4 w = s4[i];
      const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[part2 * 32 + 8 * i + 2 * e] = widen(ww[e] & 0xffffu, a.is_bf16);
        v[part2 * 32 + 8 * i + 2 * e + 1] = widen(ww[e] >> 16, a.is_bf16);
      }
    }
  }
#pragma unroll
  for (int hh = 1; hh < 32; hh *= 2) {
#pragma unroll
    for (int base = 0; base < 64; base += 2 * hh) {
#pragma unroll
      for (int i = 0; i < hh; ++i) {
        const float p = v[base + i], q = v[base + i + hh];
        v[base + i] = p + q;
        v[base + i + hh] = p - q;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    const float o = dpp_xor1(v[i]);
    v[i] = hb ? (o - v[i]) : (v[i] + o);
  }
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const float p = v[i], q = v[32 + i];
    v[i] = p + q;
    v[32 + i] = p - q;
  }
  const float c = 0.08838834764831845f;
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    v[i] = v[i] * c;
    amax = __builtin_fmaxf(amax, __builtin_fabsf(v[i]));
  }
  amax = __builtin_fmaxf(amax, dpp_xor1(amax));
  for (int j = 0; j < a.n_bits; ++j) {
    const float qm = (float)((1 << (a.bits[j] - 1)) - 1);
    const uint16_t s16 = f16_sat(amax / qm);
    const float sf = f16_to_f32(s16);
    const float inv = (sf != 0.0f) ? 1.0f / sf : 0.0f;
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < 64; ++i) {
      float r = v[i] * inv;
      r = __builtin_fminf(__builtin_fmaxf(r, -qm), qm);
      acc += sq_err(v[i], rint_i(r), sf);
    }
    acc = wave_sum(acc);
    if (lane == 0) part[j] = acc;
  }
}

__global__ void calib_reduce_kernel(CalibLaunch a) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n_comp * a.n_bits) return;
  const int comp = i / a.n_bits, j = i % a.n_bits;
  const int n_blk = a.T / kChunk;
  double s = 0.0;
  for (int b = 0; b < n_blk; ++b)
    s += a.partial[((size_t)comp * n_blk + b) * a.n_bits + j];
  a.mse[i] = s / ((double)a.T * kD);
}

}  // namespace

hipError_t launch_calibrate(const CalibLaunch& a, hipStream_t s) {
  dim3 grid(a.T / kChunk, a.n_comp);
  hipLaunchKernelGGL(calib_kernel, grid, dim3(kWave), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int n = a.n_comp * a.n_bits;
  hipLaunchKernelGGL(calib_reduce_kernel, dim3((n + 255) / 256), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace rq
