// Device helpers: number conversions, the quantizer arithmetic that decides
// codes, and the packed-chunk format (32 codes in b words; three-bit codes
// as single fields in four 24-bit quarters of a 96-bit stream, other widths
// as bit planes whose widths are the binary digits of b, codes i and i+16
// sharing the two half-words of a word).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rq {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

// Pointers into global memory.  Pointers held in a launch struct are
// generic to the compiler; accessing through a global-address-space pointer
// gives global (not flat) loads and stores, which do not tie the LDS wait
// counter to memory latency.
#define RQ_GLOBAL __attribute__((address_space(1)))
template <class T>
__device__ __forceinline__ RQ_GLOBAL T* gptr(T* p) {
  return (RQ_GLOBAL T*)p;
}

template <bool BF16>
__device__ __forceinline__ float widen_t(uint32_t bits16) {
  if constexpr (BF16) return __uint_as_float(bits16 << 16);
  const _Float16 h = __builtin_bit_cast(_Float16, (uint16_t)bits16);
  return (float)h;
}
// run-time dtype: both conversions and a select, no branch
__device__ __forceinline__ float widen(uint32_t bits16, int is_bf16) {
  const float b = widen_t<true>(bits16), f = widen_t<false>(bits16);
  return is_bf16 ? b : f;
}

// fp32 -> fp16, nearest-even, saturated at +-65504.  Returns raw bits.
__device__ __forceinline__ uint16_t f16_sat(float x) {
  x = __builtin_fminf(__builtin_fmaxf(x, -65504.0f), 65504.0f);
  return __builtin_bit_cast(uint16_t, (_Float16)x);
}

__device__ __forceinline__ float f16_to_f32(uint16_t b) {
  return (float)__builtin_bit_cast(_Float16, b);
}

// rint half-to-even of a value already clamped to [lo, hi] (|v| < 2^22).
__device__ __forceinline__ int rint_i(float v) {
  return (int)__builtin_rintf(v);
}

// Asymmetric group parameters from (min, max): zero = fp16(min), scale =
// fp16(max(max - zero, 0) / qmax); inv = 1/scale (0 when scale == 0, which
// sends every code to 0).
struct AsymParams {
  uint16_t s16, z16;
  float zf, inv;
};

__device__ __forceinline__ AsymParams asym_params(float mn, float mx,
                                                  float qmax) {
  AsymParams p;
  p.z16 = f16_sat(mn);
  p.zf = f16_to_f32(p.z16);
  float rng = __builtin_fmaxf(mx - p.zf, 0.0f);
  p.s16 = f16_sat(rng / qmax);
  float sf = f16_to_f32(p.s16);
  p.inv = (sf != 0.0f) ? 1.0f / sf : 0.0f;
  return p;
}

__device__ __forceinline__ int asym_code(float x, const AsymParams& p,
                                         float qmax) {
  float r = (x - p.zf) * p.inv;  // two roundings: built with fp-contract off
  r = __builtin_fminf(__builtin_fmaxf(r, 0.0f), qmax);
  return rint_i(r);
}

// Bit planes of a b-bit code, widest first (three-bit codes are single
// fields and do not use planes).
template <int B> struct Planes;
template <> struct Planes<1> { static constexpr int n = 1; static constexpr int w[1] = {1}; };
template <> struct Planes<2> { static constexpr int n = 1; static constexpr int w[1] = {2}; };
template <> struct Planes<4> { static constexpr int n = 1; static constexpr int w[1] = {4}; };
template <> struct Planes<5> { static constexpr int n = 2; static constexpr int w[2] = {4, 1}; };
template <> struct Planes<6> { static constexpr int n = 2; static constexpr int w[2] = {4, 2}; };
template <> struct Planes<7> { static constexpr int n = 3; static constexpr int w[3] = {4, 2, 1}; };
template <> struct Planes<8> { static constexpr int n = 1; static constexpr int w[1] = {8}; };

// Three-bit chunk: the three words are one 96-bit stream (bit 32k + j =
// bit j of word k) of four 24-bit quarters; quarter q holds codes 4q + i
// at stream bit 24q + 3i and codes 16 + 4q + i at 24q + 12 + 3i (i = 0..3).
// Codes 6 and 25 cross a word boundary.
__host__ __device__ __forceinline__ constexpr int stream3_pos(int i) {
  return 24 * ((i & 15) >> 2) + 3 * (i & 3) + (i >= 16 ? 12 : 0);
}

// Pack 32 codes (bytes, code i = byte i of c[i/4]) into B words.
template <int B>
__device__ __forceinline__ void pack_chunk(const uint32_t c[8], uint32_t out[B]) {
  if constexpr (B == 3) {
    out[0] = out[1] = out[2] = 0;
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const uint32_t code = (c[i >> 2] >> (8 * (i & 3))) & 7u;
      const int pos = stream3_pos(i), word = pos >> 5, bit = pos & 31;
      out[word] |= code << bit;
      if (bit > 29) out[word + 1] |= code >> (32 - bit);
    }
    return;
  } else {
    int word = 0, shift = 0;
#pragma unroll
    for (int p = 0; p < Planes<B>::n; ++p) {
      const int w = Planes<B>::w[p];
      const int per = 16 / w;
      const uint32_t m = (1u << w) - 1u;
#pragma unroll
      for (int d = 0; d < w; ++d) {
        uint32_t acc = 0;
#pragma unroll
        for (int k = 0; k < per; ++k) {
          const int i0 = d * per + k, i1 = 16 + d * per + k;
          uint32_t c0 = (c[i0 >> 2] >> (8 * (i0 & 3))) & 0xffu;
          uint32_t c1 = (c[i1 >> 2] >> (8 * (i1 & 3))) & 0xffu;
          acc |= ((c0 >> shift) & m) << (k * w);
          acc |= ((c1 >> shift) & m) << (16 + k * w);
        }
        out[word++] = acc;
      }
      shift += w;
    }
  }
}

// x shifted right by s bits (left when s < 0); s is a constant after
// unrolling.
__device__ __forceinline__ uint32_t shr_signed(uint32_t x, int s) {
  return s > 0 ? (x >> s) : (s < 0 ? (x << -s) : x);
}

// Entry i (wave-uniform) of a byte table held in the kernel arguments
// (4-byte aligned), read through its dword: gfx9 has no scalar byte loads,
// and a vector byte load would be waited for together with every load in
// flight before it.
__device__ __forceinline__ int kernarg_byte(const uint8_t* table, int i) {
  i = __builtin_amdgcn_readfirstlane(i);
  const uint32_t w = reinterpret_cast<const uint32_t*>(table)[i >> 2];
  return (int)((w >> (8 * (i & 3))) & 0xffu);
}

__device__ __forceinline__ h2 as_h2(uint32_t x) {
  return __builtin_bit_cast(h2, x);
}
__device__ __forceinline__ uint32_t as_u32(h2 x) {
  return __builtin_bit_cast(uint32_t, x);
}

}  // namespace rq
