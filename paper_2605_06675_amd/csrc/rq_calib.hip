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
  // orthonormal).  RTN: the same symmetric levels on the token itself.
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
  if (a.family == RQ_QUAROT) {
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
#pragma unroll
    for (int i = 0; i < 64; ++i) v[i] = v[i] * c;
  }
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < 64; ++i) amax = __builtin_fmaxf(amax, __builtin_fabsf(v[i]));
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

// ---------------------------------------------------------------- Turbo
// TurboQuant: error in the original domain, x - R^T y_hat (the bf16
// rotation is orthogonal only to about 2^-8, so the rotated-domain error
// would differ by a few percent).  One wave per (component, block):
//   y     = R x^T on bf16 (or fp16) matrix cores, fp32 sums (D[coord][token])
//   n     = |x| in fp64, t = y sqrt(128) / n, codes as in the quantizer
//   x_hat = y_hat R on fp32 matrix cores (16x16x4), k-steps taken in the
//           register order of y: step (ct, i) sums coords 16 ct + 4 g + i
// R (converted to fp32) and the block sit in LDS.
constexpr int kRRowF = 132;   // floats per LDS row of R (528 B)
constexpr int kXRow = 136;    // 16-bit entries per LDS row of the block

typedef __bf16 cbf8 __attribute__((ext_vector_type(8)));

template <int BF16>
__device__ __forceinline__ f4 mma16(u4 a, u4 b, f4 c) {
  if constexpr (BF16)
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(cbf8, a),
                                                   __builtin_bit_cast(cbf8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, a),
                                                  __builtin_bit_cast(h8, b), c, 0, 0, 0);
}

template <int B>
__device__ __forceinline__ uint32_t tcode(float t, const RQ_GLOBAL float* th) {
  constexpr int L = 1 << B, P = L / 2 - 1;
  const float m = __builtin_fabsf(t);
  int cnt = 0;
  for (int j = 0; j < P; ++j) cnt += th[j] < m ? 1 : 0;
  return (uint32_t)(t > 0.0f ? L / 2 + cnt : L / 2 - 1 - cnt);
}

template <int B>
__device__ __forceinline__ void turbo_yhat(const f4 (&y)[8][2], const float (&fs)[2],
                                           const float (&nq)[2], const float* cb,
                                           float (&yh)[8][2][4]) {
  const RQ_GLOBAL float* th = gptr(cb + (B - 1) * 512 + (1 << (B - 1)));
  const RQ_GLOBAL float* ce = gptr(cb + (B - 1) * 512 + 256);
#pragma unroll
  for (int ct = 0; ct < 8; ++ct)
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        yh[ct][tt][i] = ce[tcode<B>(y[ct][tt][i] * fs[tt], th)] * nq[tt];
}

template <int BF16>
__global__ void __launch_bounds__(kWave)
calib_turbo_kernel(CalibLaunch a) {
  __shared__ float Rf[kD * kRRowF];
  __shared__ uint16_t xs[kChunk * kXRow];
  const int blk = blockIdx.x, comp = blockIdx.y, lane = threadIdx.x;
  const int g = lane >> 4, j = lane & 15;
  const int n_blk = a.T / kChunk;
  const uint16_t* x = a.x + ((size_t)comp * a.T + (size_t)blk * kChunk) * kD;
  double* part = a.partial + ((size_t)comp * n_blk + blk) * a.n_bits;
  const uint16_t* R = a.rot + (size_t)comp * kD * kD;
  for (int e = lane; e < kD * kD / 2; e += kWave) {
    const uint32_t w = gptr(reinterpret_cast<const uint32_t*>(R))[e];
    const int r = (2 * e) / kD, c = (2 * e) % kD;
    Rf[r * kRRowF + c] = __uint_as_float(w << 16);
    Rf[r * kRRowF + c + 1] = __uint_as_float(w & 0xffff0000u);
  }
  for (int e = lane; e < kChunk * 16; e += kWave)
    *reinterpret_cast<u4*>(&xs[(e >> 4) * kXRow + 8 * (e & 15)]) =
        gptr(reinterpret_cast<const u4*>(x))[e];
  __syncthreads();
  // operands of token 16 tt + j, channels 32 ks + 8 g ..
  u4 xv[8];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      xv[4 * tt + ks] = *reinterpret_cast<const u4*>(&xs[(16 * tt + j) * kXRow + 32 * ks + 8 * g]);
  // norms
  float fs[2], nq[2];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    double s = 0.0;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const u4 w = xv[4 * tt + ks];
      const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double lo = (double)widen(ww[e] & 0xffffu, BF16);
        const double hi = (double)widen(ww[e] >> 16, BF16);
        s = __builtin_fma(lo, lo, s);
        s = __builtin_fma(hi, hi, s);
      }
    }
    s += __shfl_xor(s, 16, kWave);
    s += __shfl_xor(s, 32, kWave);
    const float nf = f16_to_f32(f16_sat((float)__builtin_sqrt(s)));
    fs[tt] = nf != 0.0f ? 11.313708498984761f / nf : 0.0f;
    nq[tt] = nf * 0.08838834764831845f;
  }
  // y = R x^T: lane holds coords 16 ct + 4 g + i of token 16 tt + j
  f4 y[8][2];
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) {
    y[ct][0] = y[ct][1] = (f4){0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      // R[16 ct + j][32 ks + 8 g ..] in the input's 16-bit type
      uint32_t rw[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float r0 = Rf[(16 * ct + j) * kRRowF + 32 * ks + 8 * g + 2 * e];
        const float r1 = Rf[(16 * ct + j) * kRRowF + 32 * ks + 8 * g + 2 * e + 1];
        uint32_t b0, b1;
        if (BF16) {
          b0 = __float_as_uint(r0) >> 16;
          b1 = __float_as_uint(r1) >> 16;
        } else {
          b0 = __builtin_bit_cast(uint16_t, (_Float16)r0);
          b1 = __builtin_bit_cast(uint16_t, (_Float16)r1);
        }
        rw[e] = b0 | (b1 << 16);
      }
      const u4 rop = {rw[0], rw[1], rw[2], rw[3]};
      y[ct][0] = mma16<BF16>(rop, xv[ks], y[ct][0]);
      y[ct][1] = mma16<BF16>(rop, xv[4 + ks], y[ct][1]);
    }
  }
  for (int jb = 0; jb < a.n_bits; ++jb) {
    float yh[8][2][4];
    switch (a.bits[jb]) {
      case 1: turbo_yhat<1>(y, fs, nq, a.cb, yh); break;
      case 2: turbo_yhat<2>(y, fs, nq, a.cb, yh); break;
      case 3: turbo_yhat<3>(y, fs, nq, a.cb, yh); break;
      case 4: turbo_yhat<4>(y, fs, nq, a.cb, yh); break;
      case 5: turbo_yhat<5>(y, fs, nq, a.cb, yh); break;
      case 6: turbo_yhat<6>(y, fs, nq, a.cb, yh); break;
      case 7: turbo_yhat<7>(y, fs, nq, a.cb, yh); break;
      default: turbo_yhat<8>(y, fs, nq, a.cb, yh); break;
    }
    // x_hat[token][channel] = sum_coord y_hat[token][coord] R[coord][channel]
    double acc = 0.0;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int nt = 0; nt < 8; ++nt) {
        f4 xh = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ct = 0; ct < 8; ++ct)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            xh = __builtin_amdgcn_mfma_f32_16x16x4f32(
                yh[ct][tt][i], Rf[(16 * ct + 4 * g + i) * kRRowF + 16 * nt + j], xh, 0, 0, 0);
        // lane: tokens 16 tt + 4 g + i, channel 16 nt + j
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float xo = widen(xs[(16 * tt + 4 * g + i) * kXRow + 16 * nt + j], BF16);
          const double d = (double)xo - (double)xh[i];
          acc = __builtin_fma(d, d, acc);
        }
      }
    acc = wave_sum(acc);
    if (lane == 0) part[jb] = acc;
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
  if (a.family == RQ_TURBO) {
    if (a.is_bf16)
      hipLaunchKernelGGL(calib_turbo_kernel<1>, grid, dim3(kWave), 0, s, a);
    else
      hipLaunchKernelGGL(calib_turbo_kernel<0>, grid, dim3(kWave), 0, s, a);
  } else {
    hipLaunchKernelGGL(calib_kernel, grid, dim3(kWave), 0, s, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int n = a.n_comp * a.n_bits;
  hipLaunchKernelGGL(calib_reduce_kernel, dim3((n + 255) / 256), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace rq
