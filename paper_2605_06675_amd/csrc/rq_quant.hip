// Quantize + pack kernels (KIVI-style, QuaRot-style and plain per-token
// symmetric RTN) and the residual window append.  One wave quantizes one 32-token block of one
// (batch entry, kv-head, K|V) unit; the unit's bit-width and code region come
// from the per-layer table in the kernel arguments.
//
// The KIVI block is staged once in LDS.  Group statistics run along one
// axis of the block and packing along the other (keys: statistics per
// channel over the 32 tokens, chunks of 32 channels per token; values: the
// reverse), so each phase reads the rows or columns it needs from LDS and
// every code goes straight into its packed word.
#include "rq_device.h"
#include "rq_internal.h"
#include "rq_ring.h"

namespace rq {

namespace {

constexpr int kWave = 64;

__device__ __forceinline__ int pair_pos(int j) {
  return j < 16 ? 2 * j : 2 * (j - 16) + 1;
}

template <int B>
__device__ __forceinline__ void store_words(uint32_t* dst, const uint32_t w[B]) {
#pragma unroll
  for (int i = 0; i < B; ++i) __builtin_nontemporal_store(w[i], dst + i);
}

template <int B>
__device__ __forceinline__ void pack_store(const uint32_t c[8], uint32_t* dst) {
  uint32_t w[B];
  pack_chunk<B>(c, w);
  store_words<B>(dst, w);
}

struct Smem {
  uint32_t codes[kChunk * kD / 4];   // [32 tokens][128 channels] bytes
  uint16_t meta[256];                // one block's metadata (512 B)
};

// ------------------------------------------------------------- KIVI (LDS)
// Persistent kernel: every wave loops over blocks (block, kv-head, batch,
// K|V in that order), with the next block's 8 KB already loading into
// registers while the current one is quantized from the wave's own LDS
// area.  The waves of a workgroup share nothing, so no
// workgroup barrier is needed: a wave's LDS operations complete in issue
// order.
constexpr int kQWaves = 4;                // waves per workgroup
constexpr int kQBuf = 1;                  // register buffers per wave
// workgroups per CU: three when every width of the layer is at most 4 bits
// (the code paths then fit 168 registers), else two
__host__ __device__ constexpr int quant_occupancy(int maxb) { return maxb <= 4 ? 3 : 2; }
constexpr int kRowW = 68;                 // dwords per staged row (272 B)
constexpr int kTabE = 34;                 // float2 entries per table row

struct KiviSmem {
  uint32_t x[kChunk * kRowW];             // [token][channel pair]
  float2 tab[4 * kTabE];                  // (zero, 1/scale): K [chunk][channel],
                                          // V [group][token]
  uint16_t meta[256];                     // the block's metadata (512 B)
};

template <int BF16>
__device__ __forceinline__ float lo16(uint32_t w) {
  if (BF16) return __uint_as_float(w << 16);
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xffffu));
}
template <int BF16>
__device__ __forceinline__ float hi16(uint32_t w) {
  if (BF16) return __uint_as_float(w & 0xffff0000u);
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
}

// Group bounds of finite inputs (minimum/maximum map to the three-input
// instructions without canonicalising every operand).
__device__ __forceinline__ float vmin(float a, float b) {
  return __builtin_elementwise_minimum(a, b);
}
__device__ __forceinline__ float vmax(float a, float b) {
  return __builtin_elementwise_maximum(a, b);
}

constexpr uint32_t kMagicBits = 0x4B000000u;   // the float 2^23

// Code of x in the low bits of a float: the clamped quotient plus 2^23 is
// rounded by the fp32 add to the nearest integer, ties to even (the
// quotient lies in [0, 2^b - 1]), leaving rint(quotient) in the low
// mantissa bits under the constant field kMagicBits.
template <int B>
__device__ __forceinline__ uint32_t kivi_code_bits(float x, float zf, float inv) {
  float r = (x - zf) * inv;               // two roundings: fp-contract is off
  r = __builtin_amdgcn_fmed3f(r, 0.0f, (float)((1 << B) - 1));
  return __float_as_uint(r + 8388608.0f);
}

// Packed words of one chunk, built by adding each code's fields at their
// bit positions.  A code arrives as kMagicBits + code; the fields of a plane
// that reaches the top bit are added as (bits >> shift), which carries the
// constant kMagicBits >> shift along, and lower planes are extracted
// exactly.  Fields never overlap, so the sum equals the OR of the fields
// plus a compile-time constant per word, removed by finish().  A three-bit
// code is one field; its part that crosses into the next word is
// (bits >> k), k <= 2, which is (kMagicBits >> k) + (code >> k) because the
// low 24 bits of kMagicBits are zero.
template <int B> struct ChunkAcc {
  uint32_t w[B];
  uint32_t bias[B];

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int i = 0; i < B; ++i) w[i] = 0, bias[i] = 0;
  }
  // code i of the chunk (0..31, constant after unrolling)
  __device__ __forceinline__ void add(int i, uint32_t cb) {
    if constexpr (B == 3) {
      const int pos = stream3_pos(i), word = pos >> 5, bit = pos & 31;
      w[word] += cb << bit;
      bias[word] += kMagicBits << bit;
      if (bit > 29) {
        w[word + 1] += cb >> (32 - bit);
        bias[word + 1] += kMagicBits >> (32 - bit);
      }
      return;
    } else {
      int word = 0, shift = 0;
#pragma unroll
      for (int p = 0; p < Planes<B>::n; ++p) {
        const int wd = Planes<B>::w[p];
        const int per = 16 / wd;
        const int j = i & 15, d = j / per, k = j % per;
        const int pos = k * wd + (i >= 16 ? 16 : 0);
        if (shift + wd == B) {
          w[word + d] += (cb >> shift) << pos;
          bias[word + d] += (kMagicBits >> shift) << pos;
        } else {
          w[word + d] += __builtin_amdgcn_ubfe(cb, shift, wd) << pos;
        }
        word += wd;
        shift += wd;
      }
    }
  }
  __device__ __forceinline__ void finish() {
#pragma unroll
    for (int i = 0; i < B; ++i) w[i] -= bias[i];
  }
};

// Code and metadata stores are non-temporal: written once per call and
// read by later calls, they need not stay in the L2 (whose dirty lines the
// end of the launch would otherwise write back).
template <int B>
__device__ __forceinline__ void store_chunk(uint32_t* dst, const uint32_t* w) {
  RQ_GLOBAL uint32_t* g = gptr(dst);
#pragma unroll
  for (int i = 0; i < B; ++i) __builtin_nontemporal_store(w[i], g + i);
}

struct BlockId {
  int blk, h, b, kind;
};

__device__ __forceinline__ BlockId block_id(const QuantLaunch& a, int it) {
  BlockId id;
  id.blk = a.blk0 + it % a.nblk;
  const int r = it / a.nblk;
  id.h = r % a.H;
  const int z = r / a.H;
  id.b = z / a.kind_n;
  id.kind = a.kind_lo + z % a.kind_n;
  return id;
}

// Global -> registers: the block's 32 token rows, 16 bytes per lane and
// step (step j, lane l: token 4 j + l / 16, bytes 16 (l % 16) of the row).
// Branch-free: each row's address selects between the new input and the
// residual window, so that every block issues the same eight loads.  The
// loads are non-temporal: every byte is read once.
__device__ __forceinline__ void load_block(const QuantLaunch& a, const BlockId& id,
                                           u4 v[8], int lane) {
  const int t0 = id.blk * kChunk;
  const uint16_t* in = (id.kind ? a.v : a.k) + (size_t)(id.b * a.H + id.h) * a.n_new * kD;
  const int cap = a.R + kChunk;
  const uint16_t* ring = a.resid + (((size_t)id.b * a.H + id.h) * 2 + id.kind) * cap * kD;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int c = j * kWave + lane, t = t0 + (c >> 4), p = c & 15;
    const uint16_t* row = t >= a.n_past ? in + (size_t)(t - a.n_past) * kD
                                        : ring + (size_t)(t % cap) * kD;
    v[j] = __builtin_nontemporal_load(gptr(reinterpret_cast<const u4*>(row)) + p);
  }
}

__device__ __forceinline__ void stage_block(KiviSmem& sm, const u4 v[8], int lane) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int c = j * kWave + lane, t = c >> 4, p = c & 15;
    *reinterpret_cast<u4*>(&sm.x[t * kRowW + 4 * p]) = v[j];
  }
  __builtin_amdgcn_wave_barrier();
}

// Metadata of the block, staged in LDS, to its 512-byte slot.
__device__ __forceinline__ void store_meta(const QuantLaunch& a, const KiviSmem& sm,
                                           const BlockId& id, int lane) {
  typedef uint32_t u2 __attribute__((ext_vector_type(2)));
  const int nblk_cap = a.cap / kChunk;
  RQ_GLOBAL u2* m = gptr(reinterpret_cast<u2*>(
      a.meta + meta_unit_offset(a.family, id.h, id.kind, id.b, a.B, nblk_cap) +
      (size_t)id.blk * kMetaBlockKivi));
  __builtin_nontemporal_store(reinterpret_cast<const u2*>(sm.meta)[lane], m + lane);
}

// Keys: scale and zero per channel over the block's 32 tokens; chunk q of
// token t holds channels 32q .. 32q + 31.
template <int BF16, int B>
__device__ __forceinline__ void kivi_keys_lds(const QuantLaunch& a, KiviSmem& sm,
                                              const BlockId& id, int lane) {
  // statistics: lane -> channels 2 lane, 2 lane + 1
  float mn0 = INFINITY, mx0 = -INFINITY, mn1 = INFINITY, mx1 = -INFINITY;
#pragma unroll
  for (int t = 0; t < kChunk; ++t) {
    const uint32_t w = sm.x[t * kRowW + lane];
    const float x0 = lo16<BF16>(w), x1 = hi16<BF16>(w);
    mn0 = vmin(mn0, x0);
    mx0 = vmax(mx0, x0);
    mn1 = vmin(mn1, x1);
    mx1 = vmax(mx1, x1);
  }
  const float qmax = (float)((1 << B) - 1);
  const AsymParams p0 = asym_params(mn0, mx0, qmax);
  const AsymParams p1 = asym_params(mn1, mx1, qmax);
  {
    const int q = lane >> 4, j = 2 * (lane & 15);
    *reinterpret_cast<float4*>(&sm.tab[q * kTabE + j]) =
        make_float4(p0.zf, p0.inv, p1.zf, p1.inv);
    sm.meta[q * 64 + pair_pos(j)] = p0.s16;
    sm.meta[q * 64 + pair_pos(j + 1)] = p1.s16;
    sm.meta[q * 64 + 32 + pair_pos(j)] = p0.z16;
    sm.meta[q * 64 + 32 + pair_pos(j + 1)] = p1.z16;
  }
  __builtin_amdgcn_wave_barrier();
  store_meta(a, sm, id, lane);
  // packing: lane -> chunk q of tokens ta and ta + 16, one token at a time
  // (the table is read twice; holding both tokens' rows costs registers)
  const int q = lane & 3, ta = lane >> 2;
  uint32_t* region = reinterpret_cast<uint32_t*>(a.codes + a.tab.code_off[id.h][0]);
  const int t0 = id.blk * kChunk;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    ChunkAcc<B> acc;
    acc.init();
    const int t = ta + 16 * u;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      __builtin_amdgcn_sched_barrier(0);
      float zf[16], inv[16];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float4 e = *reinterpret_cast<const float4*>(
            &sm.tab[q * kTabE + 16 * half + 2 * i]);
        zf[2 * i] = e.x;
        inv[2 * i] = e.y;
        zf[2 * i + 1] = e.z;
        inv[2 * i + 1] = e.w;
      }
      const u4* row = reinterpret_cast<const u4*>(&sm.x[t * kRowW + 16 * q + 8 * half]);
      const u4 d0 = row[0], d1 = row[1];
      const uint32_t w[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int i = 16 * half + 2 * k;
        acc.add(i, kivi_code_bits<B>(lo16<BF16>(w[k]), zf[2 * k], inv[2 * k]));
        acc.add(i + 1, kivi_code_bits<B>(hi16<BF16>(w[k]), zf[2 * k + 1], inv[2 * k + 1]));
      }
    }
    acc.finish();
    const size_t tok = (size_t)id.b * a.cap + t0 + t;
    store_chunk<B>(region + (tok * 4 + q) * B, acc.w);
  }
}

// Values: scale and zero per token over each group of 32 channels; chunk c
// of the block holds channel c over its 32 tokens.
template <int BF16, int B>
__device__ __forceinline__ void kivi_values_lds(const QuantLaunch& a, KiviSmem& sm,
                                                const BlockId& id, int lane) {
  const float qmax = (float)((1 << B) - 1);
  {
    // statistics: lane -> token t, groups 2 hb and 2 hb + 1
    const int t = lane >> 1, hb = lane & 1;
#pragma unroll
    for (int g2 = 0; g2 < 2; ++g2) {
      const int g = 2 * hb + g2;
      const u4* row = reinterpret_cast<const u4*>(&sm.x[t * kRowW + 16 * g]);
      float mn = INFINITY, mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const u4 d = row[i];
        const uint32_t w[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x0 = lo16<BF16>(w[e]), x1 = hi16<BF16>(w[e]);
          mn = vmin(mn, vmin(x0, x1));
          mx = vmax(mx, vmax(x0, x1));
        }
      }
      const AsymParams p = asym_params(mn, mx, qmax);
      sm.tab[g * kTabE + t] = make_float2(p.zf, p.inv);
      sm.meta[g * 64 + pair_pos(t)] = p.s16;
      sm.meta[g * 64 + 32 + pair_pos(t)] = p.z16;
    }
  }
  __builtin_amdgcn_wave_barrier();
  store_meta(a, sm, id, lane);
  // packing: lane -> channels 2 lane, 2 lane + 1 (group lane / 16)
  const int g = lane >> 4;
  ChunkAcc<B> acc0, acc1;
  acc0.init();
  acc1.init();
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    __builtin_amdgcn_sched_barrier(0);
    float zf[16], inv[16];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float4 e = *reinterpret_cast<const float4*>(
          &sm.tab[g * kTabE + 16 * half + 2 * i]);
      zf[2 * i] = e.x;
      inv[2 * i] = e.y;
      zf[2 * i + 1] = e.z;
      inv[2 * i + 1] = e.w;
    }
#pragma unroll
    for (int tt = 0; tt < 16; ++tt) {
      const int t = 16 * half + tt;
      const uint32_t w = sm.x[t * kRowW + lane];
      acc0.add(t, kivi_code_bits<B>(lo16<BF16>(w), zf[tt], inv[tt]));
      acc1.add(t, kivi_code_bits<B>(hi16<BF16>(w), zf[tt], inv[tt]));
    }
  }
  acc0.finish();
  acc1.finish();
  const int nblk_cap = a.cap / kChunk;
  uint32_t* dst = reinterpret_cast<uint32_t*>(a.codes + a.tab.code_off[id.h][1]) +
                  (((size_t)id.b * nblk_cap + id.blk) * kD + 2 * lane) * B;
  store_chunk<B>(dst, acc0.w);
  store_chunk<B>(dst + B, acc1.w);
}

template <int BF16, int MAXB>
__device__ __forceinline__ void kivi_block(const QuantLaunch& a, KiviSmem& sm,
                                           const BlockId& id, int lane) {
  const int bits = kernarg_byte(&a.tab.bits[0][0], 2 * id.h + id.kind);
#define RQ_KIVI_CASE(NB)                                          \
  case NB:                                                        \
    if (NB <= MAXB) {                                             \
      if (id.kind == 0)                                           \
        kivi_keys_lds<BF16, NB>(a, sm, id, lane);                 \
      else                                                        \
        kivi_values_lds<BF16, NB>(a, sm, id, lane);               \
    }                                                             \
    break;
  switch (bits) {
    RQ_KIVI_CASE(1)
    RQ_KIVI_CASE(2)
    RQ_KIVI_CASE(3)
    RQ_KIVI_CASE(4)
    RQ_KIVI_CASE(5)
    RQ_KIVI_CASE(6)
    RQ_KIVI_CASE(7)
    RQ_KIVI_CASE(8)
    default: break;
  }
#undef RQ_KIVI_CASE
}

// Block cur from the buffer v, whose registers then start loading the
// wave's next block.  Every step issues the same loads (past the last
// block, a copy of the last one, never used), so that the compiler's wait
// before a buffer's staging counts the younger buffers' loads on every path
// and leaves them in flight.
template <int BF16, int MAXB>
__device__ __forceinline__ void kivi_step(const QuantLaunch& a, KiviSmem& sm, int cur,
                                          int stride, int total, u4 v[8], int lane) {
  stage_block(sm, v, lane);
  const int nxt = cur + kQBuf * stride;
  load_block(a, block_id(a, nxt < total ? nxt : total - 1), v, lane);
  kivi_block<BF16, MAXB>(a, sm, block_id(a, cur), lane);
  __builtin_amdgcn_wave_barrier();
}

// MAXB: the widest bit-width of the layer (4 or 8)
template <int BF16, int MAXB>
__global__ void __launch_bounds__(kQWaves * kWave, quant_occupancy(MAXB))
kivi_quant_kernel(QuantLaunch a) {
  __shared__ KiviSmem smem[kQWaves];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & (kWave - 1);
  KiviSmem& sm = smem[wave];
  const int total = a.nblk * a.H * a.B * a.kind_n;
  const int stride = gridDim.x * kQWaves;
  int it = blockIdx.x * kQWaves + wave;
  if (a.ring_fused) copy_window(a.ring, it, stride, lane);
  if (it >= total) return;
  u4 v[8];
  load_block(a, block_id(a, it), v, lane);
  for (; it < total; it += stride) kivi_step<BF16, MAXB>(a, sm, it, stride, total, v, lane);
}

// ------------------------------------------------------- QuaRot and RTN
// Per-token symmetric quantization over the token's 128 channels; QuaRot
// (ROT = 1) first applies the orthonormal Hadamard rotation, RTN (ROT = 0)
// quantizes the vector as it is.
__device__ __forceinline__ float dpp_xor1(float v) {
  // quad_perm [1,0,3,2]: exchange with lane ^ 1
  return __builtin_bit_cast(
      float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF,
                                      0xF, true));
}

__device__ __forceinline__ float dpp_xor2(float v) {
  // quad_perm [2,3,0,1]: exchange with lane ^ 2
  return __builtin_bit_cast(
      float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF,
                                      0xF, true));
}

// One quarter of token t (channels 32 q .. 32 q + 31) into registers.
// The row address selects between the new input and the residual window
// without a branch around the loads (a divergent branch there would read
// the input pointers with vector loads and wait for every load in flight).
__device__ __forceinline__ void load_quarter(const QuantLaunch& a, int b, int h,
                                             int kind, int t, int q, u4 raw[4]) {
  const uint16_t* in = (kind ? a.v : a.k) + (size_t)(b * a.H + h) * a.n_new * kD;
  const int cap = a.R + kChunk;
  const uint16_t* ring = a.resid + (((size_t)b * a.H + h) * 2 + kind) * cap * kD;
  const uint16_t* row = t >= a.n_past ? in + (size_t)(t - a.n_past) * kD
                                      : ring + (size_t)(t % cap) * kD;
  const RQ_GLOBAL u4* s = gptr(reinterpret_cast<const u4*>(row + 32 * q));
#pragma unroll
  for (int i = 0; i < 4; ++i) raw[i] = s[i];
}

// Write this block's packed V chunks from the staged code bytes: channel c
// -> B words over the block's 32 tokens.
template <int B>
__device__ __forceinline__ void pack_values_b(const Smem& sm, uint32_t* region_blk,
                                              int lane) {
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
    pack_store<B>(w, region_blk + (size_t)c * B);
  }
}

// A block in two passes of 16 tokens; the second pass is loaded before the
// first is computed.  Lane -> token 16 p + lane / 4 and quarter q = lane % 4,
// which is exactly packed chunk q of the token.  The rotation's butterflies
// keep their order (stride 1 .. 16 inside the lane, 32 and 64 with the
// quad's lanes q ^ 1 and q ^ 2, each as one fma with a +-1 factor: the same
// single rounding of the same exact sum), so every value is the one the
// definition computes.  A code is rounded by one fp32 add of 2^23 + 2^(B-1)
// to the clamped quotient: half-to-even on the integer grid, and the even
// offset keeps the parity of ties, so the low bits hold rint(quotient) +
// 2^(B-1).
template <int ROT, int BF16, int B>
__device__ __forceinline__ void sym_block(const QuantLaunch& a, Smem& sm, int b, int h,
                                          int kind, int blk, int lane) {
  constexpr int off = 1 << (B - 1);
  constexpr float qm = (float)(off - 1);
  constexpr float magic = 8388608.0f + (float)off;
  const int t0 = blk * kChunk;
  const int tq = lane >> 2, q = lane & 3;
  uint32_t* region = reinterpret_cast<uint32_t*>(a.codes + a.tab.code_off[h][kind]);
  u4 raw[2][4];
  load_quarter(a, b, h, kind, t0 + tq, q, raw[0]);
  load_quarter(a, b, h, kind, t0 + 16 + tq, q, raw[1]);
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int t = 16 * p + tq;
    float v[32];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t ww[4] = {raw[p][i].x, raw[p][i].y, raw[p][i].z, raw[p][i].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[8 * i + 2 * e] = widen_t<BF16>(ww[e] & 0xffffu);
        v[8 * i + 2 * e + 1] = widen_t<BF16>(ww[e] >> 16);
      }
    }
    if constexpr (ROT) {
#pragma unroll
      for (int hh = 1; hh < 32; hh *= 2)
#pragma unroll
        for (int i = 0; i < 32; ++i)
          if ((i & hh) == 0) {
            const float x = v[i], y = v[i + hh];
            v[i] = x + y;
            v[i + hh] = x - y;
          }
      // stride 32: lane q ^ 1 holds channel c ^ 32; the lower half (q even)
      // takes v + o, the upper half o - v
      const float sg1 = (q & 1) ? -1.0f : 1.0f;
#pragma unroll
      for (int i = 0; i < 32; ++i) v[i] = __builtin_fmaf(sg1, v[i], dpp_xor1(v[i]));
      // stride 64: lane q ^ 2 holds channel c ^ 64
      const float sg2 = (q & 2) ? -1.0f : 1.0f;
#pragma unroll
      for (int i = 0; i < 32; ++i) v[i] = __builtin_fmaf(sg2, v[i], dpp_xor2(v[i]));
      const float c = 0.08838834764831845f;  // fp32 nearest to 1/sqrt(128)
#pragma unroll
      for (int i = 0; i < 32; ++i) v[i] = v[i] * c;
    }
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < 32; ++i) amax = __builtin_fmaxf(amax, __builtin_fabsf(v[i]));
    amax = __builtin_fmaxf(amax, dpp_xor1(amax));
    amax = __builtin_fmaxf(amax, dpp_xor2(amax));
    const uint16_t s16 = f16_sat(amax / qm);
    const float sf = f16_to_f32(s16);
    const float inv = (sf != 0.0f) ? 1.0f / sf : 0.0f;
    if (q == 0) sm.meta[pair_pos(t)] = s16;
    if (kind == 0) {
      // keys: this lane's chunk packed from registers
      ChunkAcc<B> acc;
      acc.init();
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        const float r = __builtin_amdgcn_fmed3f(v[i] * inv, -qm, qm);
        acc.add(i, __float_as_uint(r + magic));
      }
      acc.finish();
      const size_t tok = (size_t)b * a.cap + t0 + t;
      store_chunk<B>(region + (tok * 4 + q) * B, acc.w);
    } else {
      // values: code bytes staged as [token][channel] for the transpose
      uint32_t* dst = sm.codes + (t * kD) / 4 + 8 * q;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        uint32_t cb[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          cb[e] = __float_as_uint(
              __builtin_amdgcn_fmed3f(v[4 * i + e] * inv, -qm, qm) + magic);
        dst[i] = __builtin_amdgcn_perm(cb[1], cb[0], 0x0c0c0400u) |
                 __builtin_amdgcn_perm(cb[3], cb[2], 0x04000c0cu);
      }
    }
  }
  __syncthreads();
  if (kind == 1) {
    const int nblk_cap = a.cap / kChunk;
    pack_values_b<B>(sm, region + ((size_t)b * nblk_cap + blk) * kD * B, lane);
  }
}

template <int ROT, int BF16>
__global__ void __launch_bounds__(kWave)
sym_quant_kernel(QuantLaunch a) {
  __shared__ Smem sm;
  const int blk = a.blk0 + blockIdx.x;
  const int h = blockIdx.y;
  const int b = blockIdx.z / a.kind_n, kind = a.kind_lo + blockIdx.z % a.kind_n;
  const int lane = threadIdx.x;
  if (a.ring_fused)
    copy_window(a.ring, (blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x,
                gridDim.x * gridDim.y * gridDim.z, lane);
  switch (kernarg_byte(&a.tab.bits[0][0], 2 * h + kind)) {
    case 2: sym_block<ROT, BF16, 2>(a, sm, b, h, kind, blk, lane); break;
    case 3: sym_block<ROT, BF16, 3>(a, sm, b, h, kind, blk, lane); break;
    case 4: sym_block<ROT, BF16, 4>(a, sm, b, h, kind, blk, lane); break;
    case 5: sym_block<ROT, BF16, 5>(a, sm, b, h, kind, blk, lane); break;
    case 6: sym_block<ROT, BF16, 6>(a, sm, b, h, kind, blk, lane); break;
    case 7: sym_block<ROT, BF16, 7>(a, sm, b, h, kind, blk, lane); break;
    default: sym_block<ROT, BF16, 8>(a, sm, b, h, kind, blk, lane); break;
  }
  __syncthreads();
  // metadata of this block
  const int nblk_cap = a.cap / kChunk;
  uint8_t* m = a.meta + meta_unit_offset(a.family, h, kind, b, a.B, nblk_cap) +
               (size_t)blk * kMetaBlockTok;
  const uint32_t* src = reinterpret_cast<const uint32_t*>(sm.meta);
  if (lane < kMetaBlockTok / 4)
    __builtin_nontemporal_store(src[lane], reinterpret_cast<uint32_t*>(m) + lane);
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

// KIVI blocks of kinds q.kind_lo .. + q.kind_n - 1
hipError_t launch_kivi(const QuantLaunch& q, hipStream_t s) {
  int maxb = 1;
  for (int h = 0; h < q.H; ++h)
    for (int k = q.kind_lo; k < q.kind_lo + q.kind_n; ++k)
      maxb = q.tab.bits[h][k] > maxb ? q.tab.bits[h][k] : maxb;
  // persistent: as many workgroups of kQWaves waves as fit on the device
  const long waves = (long)q.nblk * q.H * q.B * q.kind_n;
  long wg = (waves + kQWaves - 1) / kQWaves;
  const long cap = (long)(q.n_cu > 0 ? q.n_cu : 256) * quant_occupancy(maxb);
  if (wg > cap) wg = cap;
  dim3 grid((unsigned)wg), block(kQWaves * kWave);
  if (maxb <= 4) {
    if (q.is_bf16)
      hipLaunchKernelGGL((kivi_quant_kernel<1, 4>), grid, block, 0, s, q);
    else
      hipLaunchKernelGGL((kivi_quant_kernel<0, 4>), grid, block, 0, s, q);
  } else {
    if (q.is_bf16)
      hipLaunchKernelGGL((kivi_quant_kernel<1, 8>), grid, block, 0, s, q);
    else
      hipLaunchKernelGGL((kivi_quant_kernel<0, 8>), grid, block, 0, s, q);
  }
  return hipGetLastError();
}

// per-token symmetric blocks (QuaRot with the rotation, RTN without) of
// kinds q.kind_lo .. + q.kind_n - 1
hipError_t launch_sym(const QuantLaunch& q, bool rot, hipStream_t s) {
  dim3 grid(q.nblk, q.H, q.B * q.kind_n);
  // bit-widths of the symmetric quantizers are 2..8 (checked on the host)
  if (rot && q.is_bf16)
    hipLaunchKernelGGL((sym_quant_kernel<1, 1>), grid, dim3(kWave), 0, s, q);
  else if (rot)
    hipLaunchKernelGGL((sym_quant_kernel<1, 0>), grid, dim3(kWave), 0, s, q);
  else if (q.is_bf16)
    hipLaunchKernelGGL((sym_quant_kernel<0, 1>), grid, dim3(kWave), 0, s, q);
  else
    hipLaunchKernelGGL((sym_quant_kernel<0, 0>), grid, dim3(kWave), 0, s, q);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize(const QuantLaunch& a, hipStream_t s) {
  if (a.nblk <= 0) return hipSuccess;
  QuantLaunch q = a;
  q.kind_lo = 0;
  q.kind_n = 2;
  if (a.family == RQ_TURBO) return launch_quantize_turbo(q, s);
  if (a.family == RQ_KIVI) return launch_kivi(q, s);
  if (a.family == RQ_KIVI_RTN) {
    // keys by KIVI, values by RTN
    q.kind_n = 1;
    hipError_t e = launch_kivi(q, s);
    if (e != hipSuccess) return e;
    q.kind_lo = 1;
    q.ring_fused = 0;   // copied by the keys' launch
    return launch_sym(q, false, s);
  }
  return launch_sym(q, a.family == RQ_QUAROT, s);
}

hipError_t launch_ring(const RingLaunch& a, hipStream_t s) {
  if (a.t_hi <= a.t_lo) return hipSuccess;
  dim3 grid(a.t_hi - a.t_lo, a.H, a.B * 2);
  hipLaunchKernelGGL(ring_kernel, grid, dim3(kWave), 0, s, a);
  return hipGetLastError();
}

}  // namespace rq
