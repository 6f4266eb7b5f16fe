// Quantize + pack kernels (KIVI-style and QuaRot-style) and the residual
// window append.  One wave quantizes one 32-token block of one
// (batch entry, kv-head, K|V) unit; the unit's bit-width and code region come
// from the per-layer table in the kernel arguments.
#include "rq_device.h"
#include "rq_internal.h"

namespace rq {

namespace {

constexpr int kWave = 64;

// Source of token t of a unit: the new input for t >= n_past, else the
// residual window.
__device__ __forceinline__ const uint16_t* token_src(const QuantLaunch& a,
                                                     int b, int h, int kind,
                                                     int t) {
  if (t >= a.n_past) {
    const uint16_t* base = kind ? a.v : a.k;
    return base + ((size_t)(b * a.H + h) * a.n_new + (t - a.n_past)) * kD;
  }
  const int cap = a.R + kChunk;
  return a.resid +
         ((((size_t)b * a.H + h) * 2 + kind) * cap + (t % cap)) * kD;
}

__device__ __forceinline__ int pair_pos(int j) {
  return j < 16 ? 2 * j : 2 * (j - 16) + 1;
}

template <int B>
__device__ __forceinline__ void store_words(uint32_t* dst, const uint32_t w[B]) {
#pragma unroll
  for (int i = 0; i < B; ++i) dst[i] = w[i];
}

template <int B>
__device__ __forceinline__ void pack_store(const uint32_t c[8], uint32_t* dst) {
  uint32_t w[B];
  pack_chunk<B>(c, w);
  store_words<B>(dst, w);
}

__device__ __forceinline__ void pack_store_dyn(int bits, const uint32_t c[8], uint32_t* dst) {
  switch (bits) {
    case 1: pack_store<1>(c, dst); break;
    case 2: pack_store<2>(c, dst); break;
    case 3: pack_store<3>(c, dst); break;
    case 4: pack_store<4>(c, dst); break;
    case 5: pack_store<5>(c, dst); break;
    case 6: pack_store<6>(c, dst); break;
    case 7: pack_store<7>(c, dst); break;
    default: pack_store<8>(c, dst); break;
  }
}

struct Smem {
  uint32_t codes[kChunk * kD / 4];   // [32 tokens][128 channels] bytes
  uint16_t meta[256];                // one block's metadata (512 B)
};

// Write this block's packed V chunks: channel c -> b words over 32 tokens.
__device__ __forceinline__ void pack_values_from_smem(const Smem& sm, int bits,
                                      uint32_t* region_blk, int lane) {
  const uint8_t* cb = reinterpret_cast<const uint8_t*>(sm.codes);
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    const int c = lane + rep * kWave;
    uint32_t w[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      w[i] = (uint32_t)cb[(4 * i + 0) * kD + c] |
             ((uint32_t)cb[(4 * i + 1) * kD + c] << 8) |
             ((uint32_t)cb[(4 * i + 2) * kD + c] << 16) |
             ((uint32_t)cb[(4 * i + 3) * kD + c] << 24);
    }
    pack_store_dyn(bits, w, region_blk + (size_t)c * bits);
  }
}

// ------------------------------------------------------------------ KIVI K
__device__ __forceinline__ void kivi_keys(const QuantLaunch& a, Smem& sm, int b, int h,
                          int blk, int lane) {
  const int bits = a.tab.bits[h][0];
  const float qmax = (float)((1 << bits) - 1);
  const int t0 = blk * kChunk;
  float x0[kChunk], x1[kChunk];
  float mn0 = INFINITY, mx0 = -INFINITY, mn1 = INFINITY, mx1 = -INFINITY;
#pragma unroll
  for (int t = 0; t < kChunk; ++t) {
    const uint32_t w =
        *reinterpret_cast<const uint32_t*>(token_src(a, b, h, 0, t0 + t) + 2 * lane);
    x0[t] = widen(w & 0xffffu, a.is_bf16);
    x1[t] = widen(w >> 16, a.is_bf16);
    mn0 = __builtin_fminf(mn0, x0[t]);
    mx0 = __builtin_fmaxf(mx0, x0[t]);
    mn1 = __builtin_fminf(mn1, x1[t]);
    mx1 = __builtin_fmaxf(mx1, x1[t]);
  }
  const AsymParams p0 = asym_params(mn0, mx0, qmax);
  const AsymParams p1 = asym_params(mn1, mx1, qmax);
  uint16_t* cs = reinterpret_cast<uint16_t*>(sm.codes);
#pragma unroll
  for (int t = 0; t < kChunk; ++t) {
    const uint32_t u0 = asym_code(x0[t], p0, qmax);
    const uint32_t u1 = asym_code(x1[t], p1, qmax);
    cs[(t * kD + 2 * lane) >> 1] = (uint16_t)(u0 | (u1 << 8));
  }
  // metadata: chunk q = lane / 16, channels j, j+1 of the chunk
  const int q = lane >> 4, j = 2 * (lane & 15);
  sm.meta[q * 64 + pair_pos(j)] = p0.s16;
  sm.meta[q * 64 + pair_pos(j + 1)] = p1.s16;
  sm.meta[q * 64 + 32 + pair_pos(j)] = p0.z16;
  sm.meta[q * 64 + 32 + pair_pos(j + 1)] = p1.z16;
  __syncthreads();
  // pack: unit (token, chunk) = lane and lane + 64
  uint32_t* region = reinterpret_cast<uint32_t*>(a.codes + a.tab.code_off[h][0]);
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    const int u = lane + rep * kWave;
    const int t = u >> 2, qq = u & 3;
    uint32_t c[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = sm.codes[(t * kD + qq * 32) / 4 + i];
    const size_t tok = (size_t)b * a.cap + t0 + t;
    pack_store_dyn(bits, c, region + (tok * 4 + qq) * bits);
  }
}

// ------------------------------------------------------------------ KIVI V
__device__ __forceinline__ void kivi_values(const QuantLaunch& a, Smem& sm, int b, int h,
                            int blk, int lane) {
  const int bits = a.tab.bits[h][1];
  const float qmax = (float)((1 << bits) - 1);
  const int t0 = blk * kChunk;
  const int t = lane >> 1, half = lane & 1;
  const uint16_t* src = token_src(a, b, h, 1, t0 + t) + half * 64;
  uint8_t* cb = reinterpret_cast<uint8_t*>(sm.codes);
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    float x[32];
    const uint4* s4 = reinterpret_cast<const uint4*>(src + g * 32);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint4 w = s4[i];
      const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[8 * i + 2 * e] = widen(ww[e] & 0xffffu, a.is_bf16);
        x[8 * i + 2 * e + 1] = widen(ww[e] >> 16, a.is_bf16);
      }
    }
    float mn = x[0], mx = x[0];
#pragma unroll
    for (int i = 1; i < 32; ++i) {
      mn = __builtin_fminf(mn, x[i]);
      mx = __builtin_fmaxf(mx, x[i]);
    }
    const AsymParams p = asym_params(mn, mx, qmax);
    uint32_t cw[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      cw[i] = (uint32_t)asym_code(x[4 * i], p, qmax) |
              ((uint32_t)asym_code(x[4 * i + 1], p, qmax) << 8) |
              ((uint32_t)asym_code(x[4 * i + 2], p, qmax) << 16) |
              ((uint32_t)asym_code(x[4 * i + 3], p, qmax) << 24);
    }
    const int cg = 2 * half + g;
    uint32_t* dst = reinterpret_cast<uint32_t*>(cb + t * kD + cg * 32);
#pragma unroll
    for (int i = 0; i < 8; ++i) dst[i] = cw[i];
    sm.meta[cg * 64 + pair_pos(t)] = p.s16;
    sm.meta[cg * 64 + 32 + pair_pos(t)] = p.z16;
  }
  __syncthreads();
  const int nblk_cap = a.cap / kChunk;
  uint32_t* region = reinterpret_cast<uint32_t*>(a.codes + a.tab.code_off[h][1]);
  pack_values_from_smem(sm, bits,
                        region + ((size_t)b * nblk_cap + blk) * kD * bits, lane);
}

// ---------------------------------------------------------------- QuaRot
__device__ __forceinline__ float dpp_xor1(float v) {
  // quad_perm [1,0,3,2]: exchange with lane ^ 1
  return __builtin_bit_cast(
      float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF,
                                      0xF, true));
}

__device__ __forceinline__ void quarot_block(const QuantLaunch& a, Smem& sm, int b, int h,
                             int kind, int blk, int lane) {
  const int bits = a.tab.bits[h][kind];
  const int off = 1 << (bits - 1);
  const float qm = (float)(off - 1);
  const int t0 = blk * kChunk;
  const int t = lane >> 1, hb = lane & 1;
  const uint16_t* src = token_src(a, b, h, kind, t0 + t);
  // v[j] = x[32 hb + j], v[32 + j] = x[64 + 32 hb + j]
  float v[64];
#pragma unroll
  for (int part = 0; part < 2; ++part) {
    const uint4* s4 = reinterpret_cast<const uint4*>(src + part * 64 + hb * 32);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint4 w = s4[i];
      const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[part * 32 + 8 * i + 2 * e] = widen(ww[e] & 0xffffu, a.is_bf16);
        v[part * 32 + 8 * i + 2 * e + 1] = widen(ww[e] >> 16, a.is_bf16);
      }
    }
  }
  // butterflies h = 1..16 inside each 32-channel run
#pragma unroll
  for (int hh = 1; hh < 32; hh *= 2) {
#pragma unroll
    for (int base = 0; base < 64; base += 2 * hh) {
#pragma unroll
      for (int i = 0; i < hh; ++i) {
        const float x = v[base + i], y = v[base + i + hh];
        v[base + i] = x + y;
        v[base + i + hh] = x - y;
      }
    }
  }
  // h = 32: partner lane holds channel + 32
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    const float o = dpp_xor1(v[i]);
    v[i] = hb ? (o - v[i]) : (v[i] + o);
  }
  // h = 64: v[j] <-> v[32 + j] in this lane
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const float x = v[i], y = v[32 + i];
    v[i] = x + y;
    v[32 + i] = x - y;
  }
  const float c = 0.08838834764831845f;  // fp32 nearest to 1/sqrt(128)
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    v[i] = v[i] * c;
    amax = __builtin_fmaxf(amax, __builtin_fabsf(v[i]));
  }
  amax = __builtin_fmaxf(amax, dpp_xor1(amax));
  const uint16_t s16 = f16_sat(amax / qm);
  const float sf = f16_to_f32(s16);
  const float inv = (sf != 0.0f) ? 1.0f / sf : 0.0f;
  uint32_t cw[2][8];
#pragma unroll
  for (int part = 0; part < 2; ++part) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      uint32_t acc = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float r = v[part * 32 + 4 * i + e] * inv;
        r = __builtin_fminf(__builtin_fmaxf(r, -qm), qm);
        acc |= (uint32_t)(rint_i(r) + off) << (8 * e);
      }
      cw[part][i] = acc;
    }
  }
  if (hb == 0) sm.meta[pair_pos(t)] = s16;
  uint32_t* region = reinterpret_cast<uint32_t*>(a.codes + a.tab.code_off[h][kind]);
  if (kind == 0) {
    // keys: chunks q = hb and 2 + hb of token t straight from registers
    const size_t tok = (size_t)b * a.cap + t0 + t;
    pack_store_dyn(bits, cw[0], region + (tok * 4 + hb) * bits);
    pack_store_dyn(bits, cw[1], region + (tok * 4 + 2 + hb) * bits);
    __syncthreads();
  } else {
    uint32_t* dst = sm.codes + (t * kD) / 4;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      dst[hb * 8 + i] = cw[0][i];
      dst[16 + hb * 8 + i] = cw[1][i];
    }
    __syncthreads();
    const int nblk_cap = a.cap / kChunk;
    pack_values_from_smem(sm, bits,
                          region + ((size_t)b * nblk_cap + blk) * kD * bits,
                          lane);
  }
}

__global__ void __launch_bounds__(kWave)
quantize_kernel(QuantLaunch a) {
  __shared__ Smem sm;
  const int blk = a.blk0 + blockIdx.x;
  const int h = blockIdx.y;
  const int b = blockIdx.z >> 1, kind = blockIdx.z & 1;
  const int lane = threadIdx.x;
  if (a.family == RQ_KIVI) {
    if (kind == 0)
      kivi_keys(a, sm, b, h, blk, lane);
    else
      kivi_values(a, sm, b, h, blk, lane);
  } else {
    quarot_block(a, sm, b, h, kind, blk, lane);
  }
  __syncthreads();
  // metadata of this block
  const int nblk_cap = a.cap / kChunk;
  const int per_blk = (a.family == RQ_KIVI) ? kMetaBlockKivi : kMetaBlockTok;
  uint8_t* m = a.meta +
               ((((size_t)h * 2 + kind) * a.B + b) * nblk_cap + blk) * per_blk;
  const int words = per_blk / 4;
  const uint32_t* src = reinterpret_cast<const uint32_t*>(sm.meta);
  for (int i = lane; i < words; i += kWave)
    reinterpret_cast<uint32_t*>(m)[i] = src[i];
}

__global__ void __launch_bounds__(kWave)
ring_kernel(RingLaunch a) {
  const int t = a.t_lo + blockIdx.x;
  const int h = blockIdx.y;
  const int b = blockIdx.z >> 1, kind = blockIdx.z & 1;
  const uint16_t* base = kind ? a.v : a.k;
  const uint32_t* src = reinterpret_cast<const uint32_t*>(
      base + ((size_t)(b * a.H + h) * a.n_new + (t - a.n_past)) * kD);
  const int cap = a.R + kChunk;
  uint32_t* dst = reinterpret_cast<uint32_t*>(
      a.resid + ((((size_t)b * a.H + h) * 2 + kind) * cap + (t % cap)) * kD);
  dst[threadIdx.x] = src[threadIdx.x];
}

}  // namespace

hipError_t launch_quantize(const QuantLaunch& a, hipStream_t s) {
  if (a.nblk <= 0) return hipSuccess;
  dim3 grid(a.nblk, a.H, a.B * 2);
  hipLaunchKernelGGL(quantize_kernel, grid, dim3(kWave), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_ring(const RingLaunch& a, hipStream_t s) {
  if (a.t_hi <= a.t_lo) return hipSuccess;
  dim3 grid(a.t_hi - a.t_lo, a.H, a.B * 2);
  hipLaunchKernelGGL(ring_kernel, grid, dim3(kWave), 0, s, a);
  return hipGetLastError();
}

}  // namespace rq
