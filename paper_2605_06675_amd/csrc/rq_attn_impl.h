// Decode attention over the packed mixed-bit cache (KIVI-style,
// QuaRot-style, TurboQuant-style and per-token symmetric RTN quantizers).
//
// Flat grid of (workgroup slot, unit) with the unit fastest, four waves per
// workgroup; a unit is one (batch, kv-head).  Slots 0 .. nwg[h]-1 stream the
// quantized 32-token blocks of their unit (about three workgroups per CU in
// all, each kv-head's share sized by the cost of its widths); the first
// slots first attend to the 16-bit residual window, 32 tokens each.  Each workgroup
// writes a partial (max, sum, acc) with cache-coherent stores and takes a
// ticket from a per-unit counter; the last to arrive merges the unit's
// partials and writes the output (QuaRot: rotated back).  A wave streams every
// fourth block of its slot's range: the block's bytes (codes and metadata)
// are fetched two blocks ahead with 1 KB-per-instruction loads and copied
// into the wave's LDS slot, from where each lane reads its MFMA operands.
//
// Per block (32 tokens) a wave runs QK^T and PV on v_mfma_f32_16x16x32_f16.
// The VALU only turns packed fields into fp16 operands: a b-bit field masked
// into mantissa bit P of a half-word whose exponent field is zero is the
// exact subnormal u * 2^(P-24) (the matrix cores keep subnormal operands),
// so one AND turns a pair of codes into a pair of operands.  The weight
// 2^(P-24) is divided out of the other operand (the query for keys, the
// probability for values) or out of the fp32 result:
//   KIVI keys    S = 2^24 sum_c (q_c s_c 2^-P) (u 2^(P-24)) + sum_c z_c q_c,
//                with q_c s_c 2^-P split into two fp16 operands (its rounded
//                value and the rounding error) so that the sum is exact
//   KIVI values  O = 2^24 sum_t (p_t s_t 2^-P) (u 2^(P-24)) + sum_t p_t z_t
//   QuaRot       per-token scales and codes u - 2^(b-1): the offset enters as
//                the accumulator's start value (keys) or one more MFMA
//                against constants (values).
//   RTN          QuaRot's path with no rotation of the query or the output.
//   TurboQuant   codes index the Lloyd-Max centroids, which are not affine
//                in the code: each pair of codes is looked up in LDS, in a
//                table of every code pair as an fp16 pair (widths 2..4, one
//                read per pair) or of the fp16 centroids (wider codes, two
//                16-bit reads); the one-bit codebook +-c is a sign OR on
//                (c, c); the per-token norm scales the scores and
//                probabilities.  The query is rotated by R on entry; the
//                merge rotates the quantized part of the output back by R^T.
// With G query heads per kv-head the sixteen MFMA columns carry the G
// queries 16/G times over; the KIVI value side uses the spare rows for the
// four 32-channel groups of a token, so one A operand serves all of them.
// Softmax runs in the log2 domain with a lazily moved maximum (it moves
// only when a block exceeds it by 2^4), so probabilities stay <= 16.
//
// Range of the fp16 operands.  Each query row is scaled by a power of two
// 2^-e so that its largest element lies in [1/2, 1); the scores are scaled
// back in fp32.  With |q 2^-e| < 1 and every scale below 65504, a key
// operand q s 2^-(P+e) stays finite.  On the value side a probability
// (<= 16) times a scale (<= 65504) can exceed the fp16 range, so each wave
// keeps a power-of-two exponent Ev (0 .. 4) by which the value operands are
// divided: it grows, like the running maximum, only when a block holds a
// scale above 4094 * 2^Ev, and the wave's value sums are rescaled then.
//

#pragma once

#include "rq_device.h"
#include "rq_internal.h"

namespace rq {

namespace {

constexpr int kWave = 64;
constexpr int kWaves = kAttnWaves;
constexpr int kThreads = kWave * kWaves;
constexpr float kInvSqrtD = 0.08838834764831845f;
constexpr uint32_t kOnes = 0x3C003C00u;    // fp16 pair (1, 1)
constexpr float kLazy = 4.0f;              // log2 headroom of the running max
// Largest value-side scale (fp16 bits) that keeps 16 * scale * 2^-Ev below
// the fp16 maximum at Ev = 0: 4094 (16 * 4094 = 65504).
constexpr uint32_t kVScaleMax = 0x6BFFu;
constexpr int kMaxEv = 4;                  // 65504 / 2^4 <= 4094

// Streaming slots per merge group (two-level merge above this).
constexpr int kGroup = kAttnGroup;
// Window tokens per window workgroup.
constexpr int kResChunk = kAttnResChunk;

// Wave priority of everything but the block loop (s_setprio operand).
constexpr int kSetupPrio = 2;
// Most LDS slots of a wave (blocks in flight).  A wave's region holds as
// many whole blocks of its unit's widths as fit, up to this many; the host
// sizes the regions so that at least two fit.
constexpr int kMaxDepth = kAttnMaxDepth;
// waves per SIMD the attention kernel is compiled for
constexpr int kAttnOcc = 3;

// ---------------------------------------------------------- field positions
// Plane widths of a b-bit code are the binary digits of b, widest first
// (three-bit codes are single fields instead: see kpair<3>).
__host__ __device__ __forceinline__ constexpr int plane_w(int b, int p) {
  int n = 0;
  for (int w = 8; w >= 1; w >>= 1)
    if (b & w) {
      if (n == p) return w;
      ++n;
    }
  return 0;
}
__host__ __device__ __forceinline__ constexpr int plane_n(int b) {
  int n = 0;
  for (int w = 8; w >= 1; w >>= 1) n += (b & w) ? 1 : 0;
  return n;
}
// first word of plane p inside a chunk == first code bit of plane p
__host__ __device__ __forceinline__ constexpr int plane_off(int b, int p) {
  int o = 0;
  for (int q = 0; q < p; ++q) o += plane_w(b, q);
  return o;
}
constexpr uint32_t pair_mask(int w) { return ((1u << w) - 1u) * 0x00010001u; }

// Key pair i (0..15) of a chunk: plane-0 slot k = i mod (16 / w0) at bit
// k * w0 of its word.  The word is shifted right by kshift before masking so
// that the whole b-bit code lies inside the 10 fp16 mantissa bits; the code
// then carries the weight 2^kpos.  One shift serves all later slots.
__host__ __device__ __forceinline__ constexpr int kshift(int b, int i) {
  const int w = plane_w(b, 0), k = i % (16 / w);
  int cur = 0;
  for (int s = 0; s <= k; ++s)
    if (s * w - cur + b > 10) cur = s * w;
  return cur;
}
__host__ __device__ __forceinline__ constexpr int kpos(int b, int i) {
  if (b == 3) return (i & 3) < 3 ? 3 * (i & 3) : 0;   // see kpair<3>
  const int w = plane_w(b, 0);
  return (i % (16 / w)) * w - kshift(b, i);
}
// Value pair slot i (0..3) of lane quarter r (codes 4r+i and 16+4r+i of a
// channel's chunk): after a per-lane pre-shift the plane-0 field sits at bit
// i * w0 (w0 <= 4), or at 8 * (i & 1) of word 2r + i/2 (w0 = 8).
__host__ __device__ __forceinline__ constexpr int vshift(int b, int i) {
  const int w = plane_w(b, 0);
  if (w == 8) return 8 * (i & 1);
  int cur = 0;
  for (int s = 0; s <= i; ++s)
    if (s * w - cur + b > 10) cur = s * w;
  return cur;
}
__host__ __device__ __forceinline__ constexpr int vpos(int b, int i) {
  if (b == 3) return i < 3 ? 3 * i : 0;               // see vpairs<3>
  const int w = plane_w(b, 0);
  return (w == 8 ? 8 * (i & 1) : i * w) - vshift(b, i);
}
// kpos and vpos of every width as a table, for set-up code where the width
// is a run-time value (the helpers above loop and divide); it travels in
// the kernel arguments, which every wave reads at its start anyway
__host__ __device__ constexpr FieldPosTab make_field_pos() {
  FieldPosTab t{};
  for (int b = 1; b <= 8; ++b) {
    for (int i = 0; i < 16; ++i) t.k[b][i] = (int8_t)kpos(b, i);
    for (int i = 0; i < 4; ++i) t.v[b][i] = (int8_t)vpos(b, i);
  }
  return t;
}

// fp16 bits of 2^-e (0 <= e <= 14), exact
constexpr uint32_t h_pow2_neg(int e) { return (uint32_t)(15 - e) << 10; }
constexpr uint32_t h_pair(uint32_t h) { return h | (h << 16); }

__device__ __forceinline__ h8 make_h8(uint32_t a, uint32_t b, uint32_t c,
                                      uint32_t d) {
  u4 v = {a, b, c, d};
  return __builtin_bit_cast(h8, v);
}
__device__ __forceinline__ h8 u4_h8(u4 v) { return __builtin_bit_cast(h8, v); }

__device__ __forceinline__ f4 mfma(h8 a, h8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float xor_shfl(float v, int mask) {
  return __shfl_xor(v, mask, kWave);
}

// max of three floats (v_maximum3_f32; the operands are never NaN, and
// fmaxf would add canonicalising moves)
__device__ __forceinline__ float max3(float a, float b, float c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}

// Wait states around the in-place rescale below: the compiler does not
// insert them for inline assembly, and its operands are MFMA results (XDL
// write -> VALU read needs up to 19) that the next MFMA reads back.
__device__ __forceinline__ void xdl_wait() {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7");
}

// x *= s in place: tying the operands keeps a rarely taken rescale from
// making the register allocator copy every accumulator on the other path
__device__ __forceinline__ void scale_inplace(f4& v, int i, float s) {
  float x = v[i];
  asm volatile("v_mul_f32 %0, %0, %1" : "+v"(x) : "v"(s));
  v[i] = x;
}

// insert the bits of x under mask into c (one v_bfi_b32; used for the
// lower planes of a code, whose bits are still zero in c)
__device__ __forceinline__ uint32_t insert(uint32_t x, uint32_t mask, uint32_t c) {
  return (x & mask) | (c & ~mask);
}

// Stores and loads of the partial results, coherent across the GPU's L2
// caches (agent scope), so that the workgroup that merges a unit's partials
// sees the other workgroups' results without a cache flush.
__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t pk_mul(uint32_t a, uint32_t b) {
  return as_u32(as_h2(a) * as_h2(b));
}

// a * b - c per fp16 half with one rounding (v_pk_fma_f16): with c the
// rounded product, the product's rounding error, exact in fp16 unless it is
// below the subnormal range
__device__ __forceinline__ uint32_t pk_fms(uint32_t a, uint32_t b, uint32_t c) {
  return as_u32(__builtin_elementwise_fma(as_h2(a), as_h2(b), -as_h2(c)));
}

// Three-bit chunks (single fields in four 24-bit quarters of the 96-bit
// stream of the chunk's words): quarter x (at bits 0..23 of x) with its
// upper 12 bits moved up by 4, so that slot s (codes 4q+s, 16+4q+s) sits
// at bits (3s, 16+3s).  Bits above 27 are left over from the neighbouring
// quarter and never selected.
__device__ __forceinline__ uint32_t spread3(uint32_t x) {
  return insert(x, 0xffffu, x << 4);
}
// quarter q (a constant after unrolling) of a chunk's three words, spread
__device__ __forceinline__ uint32_t quarter3(const uint32_t* wds, int q) {
  if (q == 0) return spread3(wds[0]);
  if (q == 1) return spread3(__builtin_amdgcn_alignbit(wds[1], wds[0], 24));
  if (q == 2) return spread3(__builtin_amdgcn_alignbit(wds[2], wds[1], 16));
  return spread3(wds[2] >> 8);
}
// quarter r (per lane) of the chunk at ch, spread: one aligned funnel
// shift of words (24r / 32, 24r / 32 + 1).  For r = 3 the second word is
// the one after the chunk; the bits taken from it land above bit 27.
__device__ __forceinline__ uint32_t lane_quarter3(const uint32_t* ch, int r) {
  const int w = (24 * r) >> 5;
  return spread3(__builtin_amdgcn_alignbit(ch[w + 1], ch[w], (24 * r) & 31));
}
// slot s of a spread quarter as a pair of fields at bits (P, 16+P), P =
// 3s for s < 3 and 0 for s = 3 (a field at bit 9 would reach the exponent)
__device__ __forceinline__ uint32_t slot3(uint32_t z, int s) {
  return s < 3 ? z & (pair_mask(3) << (3 * s)) : (z >> 9) & pair_mask(3);
}

// fp16 pair (u_i 2^(P-24), u_{i+16} 2^(P-24)) of key pair i of a chunk (its
// B words), P = kpos(B, i): the fields masked into the mantissa of a zero
// exponent, exact subnormals.
template <int B>
__device__ __forceinline__ uint32_t kpair(const uint32_t* wds, int i) {
  if constexpr (B == 3) return slot3(quarter3(wds, i >> 2), i & 3);
  constexpr int w0 = plane_w(B, 0);
  const int P = kpos(B, i);
  uint32_t acc = (wds[i / (16 / w0)] >> kshift(B, i)) & (pair_mask(w0) << P);
#pragma unroll
  for (int p = 1; p < plane_n(B); ++p) {
    const int w = plane_w(B, p), per = 16 / w, off = plane_off(B, p);
    const int pos = (i % per) * w, tgt = P + off;
    acc = insert(shr_signed(wds[off + i / per], pos - tgt), pair_mask(w) << tgt, acc);
  }
  return acc;
}

// fp16 pairs (u 2^(P-24)) of value slots i = 0..3 (codes 4r+i, 16+4r+i) of
// one channel's chunk (its B words in LDS), P = vpos(B, i).
template <int B>
__device__ __forceinline__ void vpairs(const uint32_t* ch, int r, uint32_t out[4]) {
  constexpr int w0 = plane_w(B, 0);
  if constexpr (B == 3) {
    const uint32_t z = lane_quarter3(ch, r);
#pragma unroll
    for (int i = 0; i < 4; ++i) out[i] = slot3(z, i);
  } else if constexpr (w0 == 8) {
    const uint32_t x = ch[2 * r], y = ch[2 * r + 1];
    out[0] = x & pair_mask(8);
    out[1] = (x >> 8) & pair_mask(8);
    out[2] = y & pair_mask(8);
    out[3] = (y >> 8) & pair_mask(8);
  } else {
    constexpr int per = 16 / w0;
    const uint32_t x = ch[(4 * r) / per] >> (((4 * r) % per) * w0);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      out[i] = (x >> vshift(B, i)) & (pair_mask(w0) << vpos(B, i));
#pragma unroll
    for (int p = 1; p < plane_n(B); ++p) {
      const int w = plane_w(B, p), pp = 16 / w, off = plane_off(B, p);
      const uint32_t y = ch[off + (4 * r) / pp] >> (((4 * r) % pp) * w);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tgt = vpos(B, i) + off;
        out[i] = insert(shr_signed(y, i * w - tgt), pair_mask(w) << tgt, out[i]);
      }
    }
  }
}

// ------------------------------------------------------------- TurboQuant
// Codes (i, i + 16) of a chunk as integers at bits 0 and 16 (i < 16 after
// unrolling, or, for widths other than three, a per-lane quarter base plus
// a constant).
template <int B>
__device__ __forceinline__ uint32_t tq_code_pair(const uint32_t* wds, int i) {
  // three bits: the fields at bits (0, 16); the bits above them are not
  // cleared (the caller masks)
  if constexpr (B == 3) return quarter3(wds, i >> 2) >> (3 * (i & 3));
  uint32_t f = 0;
#pragma unroll
  for (int p = 0; p < plane_n(B); ++p) {
    const int w = plane_w(B, p), per = 16 / w, off = plane_off(B, p);
    const uint32_t fld = (wds[off + i / per] >> ((i % per) * w)) & pair_mask(w);
    f |= fld << off;
  }
  return f;
}

// fp16 centroid pair of a one-bit code pair f (codes at bits 0 and 16):
// the codebook is +-c, so the pair is (c, c) with the sign bits of the
// zero codes set.  lut: the fp16 pair (c, c).
__device__ __forceinline__ uint32_t tq_lut1(uint32_t f, uint32_t lut) {
  return lut | ((~f & 0x00010001u) << 15);
}

// the fp16 pair (c, c) of the one-bit codebook from the fp32 centroid table
__device__ __forceinline__ uint32_t tq_make_lut1(const float* cb) {
  const h2 v = {(_Float16)cb[256 + 1], (_Float16)cb[256 + 1]};
  return as_u32(v);
}

// Codes (i, i + 16) of a chunk times two, at bits 1 and 17: the byte offsets
// of their entries in an fp16 table (widths 5..8).
template <int B>
__device__ __forceinline__ uint32_t tq_code2_pair(const uint32_t* wds, int i) {
  uint32_t f = 0;
#pragma unroll
  for (int p = 0; p < plane_n(B); ++p) {
    const int w = plane_w(B, p), per = 16 / w, off = plane_off(B, p);
    f |= shr_signed(wds[off + i / per], (i % per) * w - off - 1) & (pair_mask(w) << (off + 1));
  }
  return f;
}

typedef __attribute__((address_space(3))) const _Float16 lds_h;
typedef __attribute__((address_space(3))) const uint32_t lds_u32;
typedef uint16_t us2v __attribute__((ext_vector_type(2)));

// LDS tables of a TurboQuant width, one 1 KiB area per side (K, V):
// widths 2..4 hold every code pair (u, v) as the fp16 pair
// (centroid u, centroid v) at entry u + 2^b v; widths 5..8 hold the 2^b
// fp16 centroids.
constexpr int kTqTabBytes = 1024;

// fp16 centroid pair of code pair f (codes at bits 0 and 16, nothing else
// set; widths 2..4) from the pair table: the byte offset 4 u + 2^(b+2) v
// is one two-way dot product of f's halves
template <int B>
__device__ __forceinline__ uint32_t tq_tab(uint32_t f, lds_h* tab) {
  const uint32_t base = (uint32_t)(uintptr_t)tab;
  const us2v w = {4, (uint16_t)(4 << B)};
  const uint32_t off = __builtin_amdgcn_udot2(__builtin_bit_cast(us2v, f), w, base, false);
  return *(lds_u32*)(uintptr_t)off;
}

// fp16 centroid pair of a doubled code pair f from an LDS table of 2^b fp16
// centroids (widths 5..8; two 16-bit LDS reads straight into the halves)
__device__ __forceinline__ uint32_t tq_lds(uint32_t f, lds_h* tab) {
  typedef __attribute__((address_space(3))) const uint8_t lds_b;
  h2 v;
  v.x = *(lds_h*)((lds_b*)tab + (f & 0xffffu));
  v.y = *(lds_h*)((lds_b*)tab + (f >> 16));
  return as_u32(v);
}

// fp16 centroid pair of codes (i, i+16) of a chunk of width B
template <int B>
__device__ __forceinline__ uint32_t tq_pair(const uint32_t* wds, int i, uint32_t lut, lds_h* tab) {
  if constexpr (B == 1) return tq_lut1(tq_code_pair<B>(wds, i), lut);
  else if constexpr (B <= 4) return tq_tab<B>(tq_code_pair<B>(wds, i) & pair_mask(B), tab);
  else return tq_lds(tq_code2_pair<B>(wds, i), tab);
}

// Key-side and value-side paths of a family.  The mixed family (KIVI keys,
// RTN values) takes the KIVI path for its keys and the per-token symmetric
// path (the QuaRot instantiation, queries left unrotated) for its values.
__host__ __device__ constexpr int key_fam(int f) { return f == RQ_KIVI_RTN ? RQ_KIVI : f; }
__host__ __device__ constexpr int val_fam(int f) { return f == RQ_KIVI_RTN ? RQ_QUAROT : f; }

// ------------------------------------------------------------ wave state
template <int NA>
struct WaveState {
  f4 acc[8];        // PV accumulators, channel tiles 16nt..16nt+15, scaled by
                    // 2^-(24+Ev) (codes as subnormals) or 2^-Ev (TurboQuant)
  f4 corrO;         // QuaRot/RTN: sum_t p s 2^-Ev (the symmetric offset term)
  f4 corrZ;         // KIVI: sum_t p z_{t,g} in column g, sum_t p in column 4;
                    // others: sum_t p in every column
  float m_run;      // running max of this lane's query (log2 domain)
  int ev;           // value-side exponent Ev (the same in every lane)
  uint32_t wv[4];   // fp16 pair 2^-(vpos(i) + Ev) of value slot i
                    // (TurboQuant: 2^-Ev)
};

// Static per-lane operands built once per workgroup.
struct LaneOps {
  uint32_t qh[16];  // QK B operand: fp16 q' 2^-(kpos + e) per k-slot pair
                    // (TurboQuant: q' 2^-e), q' the query (QuaRot: H q /
                    // sqrt(128), TurboQuant: R q / sqrt(128))
  uint32_t qz[16];  // KIVI: fp16 q' 2^-e per k-slot pair (zero-point term)
  uint32_t vq[4];   // QuaRot/RTN: fp16 pair 2^vpos(i) of value slot i
  f4 corrK;         // QuaRot/RTN: -2^(b-1) sum_c 2^(kpos-24) qh (start value
                    // of the score accumulators; the same in all rows)
  float cK;         // qscale 2^(24+e) (codes as subnormals) or qscale 2^e
                    // (TurboQuant), qscale = scale * log2(e)
  float eK;         // KIVI: qscale 2^e (the zero-point sum)
  uint32_t lut1;    // TurboQuant: the fp16 pair (c, c) of the one-bit
                    //   codebook +-c
  lds_h* tabk;      // TurboQuant: LDS tables of the K and V widths (pairs
  lds_h* tabv;      //   for widths 2..4; centroids for widths >= 5)
  int r, col, lane;
  int gsub;         // col / GP
  int GP;           // queries per replica (power of two >= G)
};

struct SlotPtrs {
  const uint32_t* kc;  // K codes of the block (LDS)
  const uint32_t* vc;  // V codes
  const u4* km;        // K metadata
  const u4* vm;        // V metadata
};

// K side of one block: t0 (tokens 4r+i), t1 (tokens 16+4r+i), the log2
// scores of this lane's query relative to m_ref.  A operands: tile t
// (tokens 16t..16t+15, row = col), k-slot pairs (kb, k') of chunk r,
// unpacked per K-step.
template <int FAM, int BK>
__device__ __forceinline__ void kpart(const SlotPtrs& sp, const LaneOps& lo, float m_ref,
                                      f4& t0, f4& t1) {
  const int r = lo.r;
  uint32_t kw[2][BK];
#pragma unroll
  for (int tile = 0; tile < 2; ++tile)
#pragma unroll
    for (int i = 0; i < BK; ++i) kw[tile][i] = sp.kc[((16 * tile + lo.col) * 4 + r) * BK + i];
  f4 S0, S1;
  if constexpr (FAM == RQ_KIVI) {
    // per-channel scales folded into the query as an exact fp16 pair
    // hi + lo = q' s 2^-(kpos+e) (hi the rounded product, lo its rounding
    // error), both against the same codes; the zero points enter through
    // their own chain X = sum_c z_c q'_c 2^-e, the same in all rows
    f4 X = {0.f, 0.f, 0.f, 0.f};
    S0 = X;
    S1 = X;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const u4 s4 = sp.km[r * 8 + kb], z4 = sp.km[r * 8 + 4 + kb];
      const uint32_t s[4] = {s4.x, s4.y, s4.z, s4.w};
      uint32_t hi[4], lw[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        hi[i] = pk_mul(lo.qh[4 * kb + i], s[i]);
        lw[i] = pk_fms(lo.qh[4 * kb + i], s[i], hi[i]);
      }
      const h8 Bhi = make_h8(hi[0], hi[1], hi[2], hi[3]);
      const h8 Blo = make_h8(lw[0], lw[1], lw[2], lw[3]);
      X = mfma(u4_h8(z4), make_h8(lo.qz[4 * kb], lo.qz[4 * kb + 1], lo.qz[4 * kb + 2],
                                  lo.qz[4 * kb + 3]), X);
      const h8 A0 = make_h8(kpair<BK>(kw[0], 4 * kb), kpair<BK>(kw[0], 4 * kb + 1),
                            kpair<BK>(kw[0], 4 * kb + 2), kpair<BK>(kw[0], 4 * kb + 3));
      const h8 A1 = make_h8(kpair<BK>(kw[1], 4 * kb), kpair<BK>(kw[1], 4 * kb + 1),
                            kpair<BK>(kw[1], 4 * kb + 2), kpair<BK>(kw[1], 4 * kb + 3));
      S0 = mfma(A0, Bhi, S0);
      S1 = mfma(A1, Bhi, S1);
      S0 = mfma(A0, Blo, S0);
      S1 = mfma(A1, Blo, S1);
    }
    const float xx = __builtin_fmaf(X[0], lo.eK, -m_ref);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      t0[i] = __builtin_fmaf(S0[i], lo.cK, xx);
      t1[i] = __builtin_fmaf(S1[i], lo.cK, xx);
    }
  } else {
    S0 = FAM == RQ_TURBO ? (f4){0.f, 0.f, 0.f, 0.f} : lo.corrK;
    S1 = S0;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const h8 Bk = make_h8(lo.qh[4 * kb], lo.qh[4 * kb + 1], lo.qh[4 * kb + 2],
                            lo.qh[4 * kb + 3]);
      if constexpr (FAM == RQ_TURBO) {
        S0 = mfma(make_h8(tq_pair<BK>(kw[0], 4 * kb, lo.lut1, lo.tabk),
                          tq_pair<BK>(kw[0], 4 * kb + 1, lo.lut1, lo.tabk),
                          tq_pair<BK>(kw[0], 4 * kb + 2, lo.lut1, lo.tabk),
                          tq_pair<BK>(kw[0], 4 * kb + 3, lo.lut1, lo.tabk)),
                  Bk, S0);
        S1 = mfma(make_h8(tq_pair<BK>(kw[1], 4 * kb, lo.lut1, lo.tabk),
                          tq_pair<BK>(kw[1], 4 * kb + 1, lo.lut1, lo.tabk),
                          tq_pair<BK>(kw[1], 4 * kb + 2, lo.lut1, lo.tabk),
                          tq_pair<BK>(kw[1], 4 * kb + 3, lo.lut1, lo.tabk)),
                  Bk, S1);
      } else {
        S0 = mfma(make_h8(kpair<BK>(kw[0], 4 * kb), kpair<BK>(kw[0], 4 * kb + 1),
                          kpair<BK>(kw[0], 4 * kb + 2), kpair<BK>(kw[0], 4 * kb + 3)),
                  Bk, S0);
        S1 = mfma(make_h8(kpair<BK>(kw[1], 4 * kb), kpair<BK>(kw[1], 4 * kb + 1),
                          kpair<BK>(kw[1], 4 * kb + 2), kpair<BK>(kw[1], 4 * kb + 3)),
                  Bk, S1);
      }
    }
    // per-token scales (TurboQuant: norms): dword 4r+i of the pair-ordered
    // scales holds tokens (4r+i, 16+4r+i)
    const u4 sv = sp.km[r];
    const uint32_t ss[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const h2 sc = as_h2(ss[i]);
      t0[i] = __builtin_fmaf(S0[i] * lo.cK, (float)sc.x, -m_ref);
      t1[i] = __builtin_fmaf(S1[i] * lo.cK, (float)sc.y, -m_ref);
    }
  }
}

// The value-side scales this lane multiplies into its A operands (KIVI: the
// groups of its A operands; others: the per-token scales or norms), as
// fp16 pairs.
template <int FAM, int NA>
struct VScales {
  u4 s[FAM == RQ_KIVI ? NA : 1];
};

template <int FAM, int NA>
__device__ __forceinline__ VScales<FAM, NA> load_vscales(const SlotPtrs& sp, const LaneOps& lo) {
  VScales<FAM, NA> v;
  if constexpr (FAM == RQ_KIVI) {
    constexpr int GPA = 4 / NA;   // value groups per A operand
#pragma unroll
    for (int a = 0; a < NA; ++a) v.s[a] = sp.vm[(a * GPA + lo.gsub % GPA) * 8 + lo.r];
  } else {
    v.s[0] = sp.vm[lo.r];
  }
  return v;
}

typedef uint16_t us2 __attribute__((ext_vector_type(2)));

// Largest of the lane's value-side scales as an fp16 pair (both halves are
// candidates; the scales are >= 0, so their bit patterns order like them).
template <int FAM, int NA>
__device__ __forceinline__ us2 vscale_max(const VScales<FAM, NA>& v) {
  constexpr int n = FAM == RQ_KIVI ? NA : 1;
  us2 m = __builtin_bit_cast(us2, v.s[0].x);
#pragma unroll
  for (int a = 0; a < n; ++a) {
    if (a > 0) m = __builtin_elementwise_max(m, __builtin_bit_cast(us2, v.s[a].x));
    m = __builtin_elementwise_max(m, __builtin_bit_cast(us2, v.s[a].y));
    m = __builtin_elementwise_max(m, __builtin_bit_cast(us2, v.s[a].z));
    m = __builtin_elementwise_max(m, __builtin_bit_cast(us2, v.s[a].w));
  }
  return m;
}

// V side of one block: probabilities P (fp16 pairs of tokens 4r+i and
// 16+4r+i of this lane's query) times the dequantized values; B operands:
// tile nt (channels 16nt..16nt+15, column = col), token slots of quarter r.
template <int FAM, int NA, int BV>
__device__ __forceinline__ void vpart(const SlotPtrs& sp, const LaneOps& lo,
                                      const uint32_t (&P)[4], const VScales<FAM, NA>& vs,
                                      const uint32_t* cst, WaveState<NA>& ws) {
  constexpr int GPA = 4 / NA;   // value groups per A operand (KIVI)
  const int r = lo.r, col = lo.col;
  uint32_t P2[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) P2[i] = pk_mul(P[i], ws.wv[FAM == RQ_TURBO ? 0 : i]);
  constexpr int nA = FAM == RQ_KIVI ? NA : 1;
  uint32_t A[nA][4];
#pragma unroll
  for (int a = 0; a < nA; ++a) {
    A[a][0] = pk_mul(P2[0], vs.s[a].x);
    A[a][1] = pk_mul(P2[1], vs.s[a].y);
    A[a][2] = pk_mul(P2[2], vs.s[a].z);
    A[a][3] = pk_mul(P2[3], vs.s[a].w);
  }
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) {
    const int a = (FAM == RQ_KIVI) ? (nt / 2) / GPA : 0;
    uint32_t pr[4];
    if constexpr (FAM == RQ_TURBO) {
      const uint32_t* ch = sp.vc + (16 * nt + col) * BV;
      if constexpr (BV == 3) {
        const uint32_t z = lane_quarter3(ch, r);
#pragma unroll
        for (int i = 0; i < 4; ++i) pr[i] = tq_tab<3>((z >> (3 * i)) & pair_mask(3), lo.tabv);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) pr[i] = tq_pair<BV>(ch, 4 * r + i, lo.lut1, lo.tabv);
      }
    } else {
      vpairs<BV>(sp.vc + (16 * nt + col) * BV, r, pr);
    }
    ws.acc[nt] = mfma(make_h8(A[a][0], A[a][1], A[a][2], A[a][3]),
                      make_h8(pr[0], pr[1], pr[2], pr[3]), ws.acc[nt]);
  }
  const h8 Ph = make_h8(P[0], P[1], P[2], P[3]);
  if constexpr (FAM == RQ_KIVI) {
    // column g < 4: zero points of group g; column 4: ones; others: zeros
    const u4 bz = (col < 4) ? sp.vm[col * 8 + 4 + r]
                            : reinterpret_cast<const u4*>(cst)[col == 4 ? 0 : 1];
    ws.corrZ = mfma(Ph, u4_h8(bz), ws.corrZ);
  } else {
    if constexpr (FAM != RQ_TURBO)
      ws.corrO = mfma(make_h8(A[0][0], A[0][1], A[0][2], A[0][3]),
                      make_h8(lo.vq[0], lo.vq[1], lo.vq[2], lo.vq[3]), ws.corrO);
    ws.corrZ = mfma(Ph, make_h8(kOnes, kOnes, kOnes, kOnes), ws.corrZ);
  }
}

// fp16 pairs 2^-(vpos(i) + ev) of the value slots (TurboQuant: 2^-ev)
template <int FAM, int BV>
__device__ __forceinline__ void set_wv(int ev, uint32_t wv[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int e = (FAM == RQ_TURBO ? 0 : vpos(BV, i)) + ev;
    wv[i] = h_pair((uint32_t)(15 - e) << 10);
  }
}

// The rarely taken part of a block: move the running maximum of the lane's
// query to the block's, and/or raise the value exponent Ev until every
// value-side scale of the block is at most 4094 * 2^Ev; rescale the wave's
// sums accordingly.
template <int FAM, int NA, int BV>
__device__ __forceinline__ void block_rescale(const LaneOps& lo, float m_ref, float mx,
                                              us2 smax, f4& t0, f4& t1, WaveState<NA>& ws) {
  mx = __builtin_fmaxf(mx, xor_shfl(mx, 16));
  mx = __builtin_fmaxf(mx, xor_shfl(mx, 32));
  const float mnew = __builtin_fmaxf(ws.m_run, m_ref + mx);
  const float alpha = __builtin_amdgcn_exp2f(ws.m_run - mnew);
  const float delta = m_ref - mnew;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    t0[i] += delta;
    t1[i] += delta;
  }
  ws.m_run = mnew;
  // exponent this lane's scales need, then the wave's
  const int sb = smax.x > smax.y ? smax.x : smax.y;
  int need = sb > (int)kVScaleMax ? (sb - (int)kVScaleMax + 1023) >> 10 : 0;
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    const int o = __shfl_xor(need, d, kWave);
    need = o > need ? o : need;
  }
  const int ev_new = need > ws.ev ? need : ws.ev;
  const float fv = __builtin_ldexpf(1.0f, ws.ev - ev_new);
  if (ev_new != ws.ev) {
    ws.ev = ev_new;
    set_wv<FAM, BV>(ev_new, ws.wv);
  }
  xdl_wait();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // accumulator row 4r+i belongs to query (4r+i) mod GP
    const float ar = __shfl(alpha, (4 * lo.r + i) & (lo.GP - 1), kWave);
    const float av = ar * fv;
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) scale_inplace(ws.acc[nt], i, av);
    if constexpr (FAM == RQ_QUAROT) scale_inplace(ws.corrO, i, av);
    scale_inplace(ws.corrZ, i, ar);
  }
  xdl_wait();
}

// One block from the LDS slot: QK^T, online softmax, PV.
template <int FAM, int NA, int BK, int BV>
__device__ __forceinline__ void block_step(const uint8_t* slot, const LaneOps& lo,
                                           const uint32_t* cst, WaveState<NA>& ws) {
  constexpr int KF = key_fam(FAM), VF = val_fam(FAM);
  constexpr int MBK = meta_block_bytes(FAM, 0);
  SlotPtrs sp;
  sp.kc = reinterpret_cast<const uint32_t*>(slot);
  sp.vc = reinterpret_cast<const uint32_t*>(slot + 512 * BK);
  sp.km = reinterpret_cast<const u4*>(slot + 512 * (BK + BV));
  sp.vm = reinterpret_cast<const u4*>(slot + 512 * (BK + BV) + MBK);
  const float m_ref = ws.m_run == -INFINITY ? 0.0f : ws.m_run;
  f4 t0, t1;
  kpart<KF, BK>(sp, lo, m_ref, t0, t1);
  const VScales<VF, NA> vs = load_vscales<VF, NA>(sp, lo);
  // keep the phases apart: hoisting all LDS reads of the block to its top
  // needs more registers than the waves per SIMD allow
  __builtin_amdgcn_sched_barrier(0);
  float mx = max3(t0[0], t1[0], t0[1]);
  mx = max3(mx, t1[1], t0[2]);
  mx = max3(mx, t1[2], t0[3]);
  mx = max3(mx, t1[3], t1[3]);
  const us2 smax = vscale_max<VF, NA>(vs);
  const uint32_t thr = (kVScaleMax + ((uint32_t)ws.ev << 10)) * 0x00010001u;
  const bool big = __builtin_bit_cast(uint32_t, __builtin_elementwise_max(
                       smax, __builtin_bit_cast(us2, thr))) != thr;
  if (__builtin_amdgcn_ballot_w64(!(mx <= kLazy) || ws.m_run == -INFINITY || big))
    block_rescale<VF, NA, BV>(lo, m_ref, mx, smax, t0, t1, ws);
  uint32_t P[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const h2 pv = {(_Float16)__builtin_amdgcn_exp2f(t0[i]),
                   (_Float16)__builtin_amdgcn_exp2f(t1[i])};
    P[i] = as_u32(pv);
  }
  __builtin_amdgcn_sched_barrier(0);
  vpart<VF, NA, BV>(sp, lo, P, vs, cst, ws);
}

// A block's data is four contiguous byte ranges: K codes (512*BK), V codes
// (512*BV), K metadata and V metadata (the family's metadata bytes of a
// block of each kind).  A wave copies it straight from global memory into
// one of its LDS slots with buffer_load_dwordx4 .. lds: piece k of lane l
// covers bytes [16 l + 1024 k, +16) of the concatenation, so every
// instruction moves up to 1 KB of contiguous memory and no VGPR holds the
// data in flight.  Two buffer resources per unit: its codes (K then V,
// based at its K codes) and its metadata (based at its K metadata); the
// piece that holds the end of the codes and the start of the metadata takes
// one instruction for each.  (The flat-encoded global_load_lds would do
// the same copies, but the compiler's wait insertion counts it as an LDS
// access as well and then waits for every LDS read in flight before using
// any of them.)
template <int FAM, int BK, int BV> struct Slot {
  static constexpr int kb = 512 * BK;
  static constexpr int vb = 512 * BV;
  static constexpr int cb = kb + vb;            // code bytes
  static constexpr int kmb = meta_block_bytes(FAM, 0);
  static constexpr int vmb = meta_block_bytes(FAM, 1);
  static constexpr int bytes = cb + kmb + vmb;
  static constexpr int pieces = (bytes + 1023) / 1024;
  static constexpr int ops = pieces + (cb % 1024 != 0 ? 1 : 0);   // copy instructions
};

struct Geo {
  __amdgpu_buffer_rsrc_t codes;  // this unit's K codes, then (at voff) its V codes
  __amdgpu_buffer_rsrc_t meta;   // its K metadata, then (at vmoff) its V metadata
  uint32_t voff, vmoff;
};

// Buffer resource over n bytes at p (raw 32-bit data format, no swizzle;
// accesses at or beyond n read zeros).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void* p, uint32_t n) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)n, 0x00020000);
}

typedef __attribute__((address_space(3))) void lds_void;

// Cache policy of the block copies: non-temporal (the NT bit), so that the
// cache blocks streamed once per call are the first to leave the L2 and
// the kernel's code and small shared data stay there across calls.
constexpr int kStreamPolicy = 2;

// Piece k of block blk into slot (lane: this lane's 16 bytes at o).
__device__ __forceinline__ void copy_piece(const Geo& g, int blk, int o, int kb, int vb, int cb,
                                           int kmb, int vmb, int bytes, bool has_codes,
                                           bool has_meta, lds_void* dst) {
  const uint32_t ub = (uint32_t)blk;
  if (has_codes && o < cb) {
    const uint32_t off = o < kb ? ub * kb + o : g.voff + ub * vb + (o - kb);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(g.codes, dst, 16, off, 0, 0, kStreamPolicy);
  }
  if (has_meta && o >= cb && o < bytes) {
    const int m = o - cb;
    const uint32_t off = m < kmb ? ub * kmb + m : g.vmoff + ub * vmb + (m - kmb);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(g.meta, dst, 16, off, 0, 0, kStreamPolicy);
  }
}

template <int FAM, int BK, int BV>
__device__ __forceinline__ void issue_block(const Geo& g, int blk, int lane, uint8_t* slot) {
  using S = Slot<FAM, BK, BV>;
#pragma unroll
  for (int k = 0; k < S::pieces; ++k)
    copy_piece(g, blk, 16 * lane + 1024 * k, S::kb, S::vb, S::cb, S::kmb, S::vmb, S::bytes,
               1024 * k < S::cb, 1024 * (k + 1) > S::cb, (lds_void*)(slot + 1024 * k));
}

// Wait until at most N vector-memory operations of this wave are in flight
// (gfx9 s_waitcnt encoding: vmcnt in bits 3:0 and 15:14, expcnt and lgkmcnt
// at their maxima).  The compiler does not track LDS written by the
// buffer-to-LDS copies, so the reads of a slot are fenced by hand.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
  asm volatile("" ::: "memory");
}

// Static blocks j0 .. j1-1 of a wave's ring (block blk0 + j stride, below
// nblk, into slot j at j * bytes; the layout of Slot<> at run time).
// Returns the copy instructions issued.
__device__ __forceinline__ int issue_first(const Geo& g, int bk, int bv, int mk, int mv, int j0,
                                           int j1, int blk0, int stride, int nblk, int lane,
                                           uint8_t* slots) {
  const int kb = 512 * bk, vb = 512 * bv, cb = kb + vb, bytes = cb + mk + mv;
  const int pieces = (bytes + 1023) / 1024;
  const int ops = pieces + (cb % 1024 != 0 ? 1 : 0);
  int issued = 0;
  for (int j = j0; j < j1; ++j) {
    const int blk = blk0 + stride * j;
    if (blk >= nblk) break;
    issued += ops;
    uint8_t* slot = slots + j * bytes;
    for (int k = 0; k < pieces; ++k)
      copy_piece(g, blk, 16 * lane + 1024 * k, kb, vb, cb, mk, mv, bytes, 1024 * k < cb,
                 1024 * (k + 1) > cb, (lds_void*)(slot + 1024 * k));
  }
  return issued;
}

// wait_vm<n> for a run-time n (0 .. 31; larger counts wait for everything)
__device__ __forceinline__ void wait_vm_rt(int n) {
  switch (n) {
#define RQ_W(N) case N: wait_vm<N>(); break;
    RQ_W(1) RQ_W(2) RQ_W(3) RQ_W(4) RQ_W(5) RQ_W(6) RQ_W(7) RQ_W(8) RQ_W(9) RQ_W(10)
    RQ_W(11) RQ_W(12) RQ_W(13) RQ_W(14) RQ_W(15) RQ_W(16) RQ_W(17) RQ_W(18) RQ_W(19)
    RQ_W(20) RQ_W(21) RQ_W(22) RQ_W(23) RQ_W(24) RQ_W(25) RQ_W(26) RQ_W(27) RQ_W(28)
    RQ_W(29) RQ_W(30) RQ_W(31)
#undef RQ_W
    default: wait_vm<0>(); break;
  }
}

// The wait before a block of P copy instructions, n the operations issued
// after its copies: the largest multiple of P + 1 not above n (waiting for
// fewer outstanding operations is always safe).  In steady state n is
// (depth - 1) (P + 1) (the later slots' copies and claims) and the wait
// exact; the other values occur while the ring fills, when the operations
// it also waits for were issued right after the slot's.  Three compares at
// most, so that the loop does not walk a search tree per block.
template <int P>
__device__ __forceinline__ void wait_slot(int n) {
  if (n >= 3 * (P + 1)) wait_vm<3 * (P + 1)>();
  else if (n >= 2 * (P + 1)) wait_vm<2 * (P + 1)>();
  else if (n >= P + 1) wait_vm<P + 1>();
  else wait_vm<0>();
}

// The wait for a claim with n operations issued after it: the largest
// multiple of P (the copies of one block) not above n.
template <int P>
__device__ __forceinline__ void wait_claim(int n) {
  if (n >= 4 * P) wait_vm<4 * P>();
  else if (n >= 3 * P) wait_vm<3 * P>();
  else if (n >= 2 * P) wait_vm<2 * P>();
  else if (n >= P) wait_vm<P>();
  else wait_vm<0>();
}

// Arrival and claim counters (agent scope, 64 bits): the upper half holds
// the number of the call counting in it (the host numbers the calls on a
// workspace 1, 2, ..), the lower half the count.  The last user of a
// counter in a call leaves (next number, 0), so the next call on the
// workspace finds its counters ready; a counter with another tag (a zeroed
// workspace, or a count left by a call that did not finish) is stale, and
// the first arrival of the call takes it over.
__device__ __forceinline__ uint32_t next_epoch(uint32_t e) { return e + 1u == 0u ? 1u : e + 1u; }

__device__ __forceinline__ uint64_t ctr_add(uint64_t* c) {
  return __hip_atomic_fetch_add(c, (uint64_t)1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The count an arrival took, from its fetch-add result `old` (one lane).
// With a stale tag the add does not count: the arrival installs
// (epoch, 1), taking count 0, unless another arrival installed the tag
// first, and then adds again.  Every turn of the loop returns or follows a
// change of the counter by another arrival, and an arrival changes it at
// most twice, so the loop ends.
__device__ __forceinline__ uint32_t ctr_count(uint64_t* c, uint64_t old, uint32_t epoch) {
  if ((uint32_t)(old >> 32) == epoch) return (uint32_t)old;
  const uint64_t first = ((uint64_t)epoch << 32) | 1u;
  for (;;) {
    uint64_t cur = __hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((uint32_t)(cur >> 32) == epoch) {
      const uint64_t o = ctr_add(c);
      if ((uint32_t)(o >> 32) == epoch) return (uint32_t)o;
    } else if (__hip_atomic_compare_exchange_strong(c, &cur, first, __ATOMIC_RELAXED,
                                                    __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT)) {
      return 0;
    }
  }
}

// Block claims of a wave: the unit's blocks beyond the statically assigned
// first ones go to whichever wave asks next (an agent-scope counter), so
// that waves and workgroups that run faster take more of them.
struct Claims {
  uint64_t* ctr;       // the unit's claim counter
  int base;            // first dynamically assigned block
  int nblk;            // blocks of the unit
  uint32_t epoch;      // the call's tag
  int mark;            // the wave's operation count just after the claim
  bool live;           // a claim is in flight
};

// The claim's fetch-add returns into v[166:167] of lane 0, registers
// written and read only by these inline statements: the kernel leaves them
// out of the compiler's allocation (and the build rejects attention code in
// which the compiler uses them itself).
// The compiler's wait insertion does not order the LDS-DMA block copies
// with other loads, so a result in a register it tracks would be waited
// for with every copy in flight; here the wave waits itself, for the claim
// and what was issued before it (claim_take).
#define RQ_CLAIM_REGS "memory", "v166", "v167"

__device__ __forceinline__ void claim_issue(uint64_t* ctr, int lane) {
  if (lane == 0)
    asm volatile("global_atomic_add_x2 v[166:167], %0, %1, off sc0" ::"v"(ctr),
                 "v"((uint64_t)1) : RQ_CLAIM_REGS);
}

// The claimed index (relative to cl.base); n: the operations this wave
// issued after the claim.
template <int P>
__device__ __forceinline__ int claim_take(const Claims& cl, int lane, int n) {
  wait_claim<P>(n);
  uint32_t lo, hi;
  asm volatile("v_mov_b32 %0, v166\n\tv_mov_b32 %1, v167" : "=v"(lo), "=v"(hi) :: RQ_CLAIM_REGS);
  uint32_t v = 0;
  if (lane == 0) v = ctr_count(cl.ctr, ((uint64_t)hi << 32) | lo, cl.epoch);
  return __builtin_amdgcn_readfirstlane((int)v);
}

// The wave's blocks, up to `depth` (2 .. kMaxDepth) in flight in a ring of
// slots of the block's exact size.  Its n_static statically assigned blocks
// (blk0 + j stride into slot j) come first: the prologue issued the first
// n_up (the whole ring: the first before the set-up, the others right after
// it, so that memory stays busy while the first blocks are computed), any
// others follow one per computed block.  Then claimed blocks:
// each slot is refilled after it has been computed; the claim for the
// block after that is issued just before the refill, so its result has a
// whole block's time to come back.  `issued` counts this wave's
// vector-memory operations (copies and claims) so that the wait for a slot
// leaves everything issued after it in flight.  Claims exist only when all
// `depth` slots receive a static block, so blocks are always consumed in
// ring order.
template <int FAM, int NA, int BK, int BV>
__device__ __forceinline__ void stream_blocks(const Geo& g, int depth, int n_static, int n_up,
                                              int blk0, int stride, Claims& cl, int issued,
                                              uint8_t* slots, const LaneOps& lo,
                                              const uint32_t* cst, WaveState<NA>& ws) {
  using S = Slot<FAM, BK, BV>;
  static_assert(kMaxDepth == 4, "the ring below rotates four marks");
  // m0: `issued` just after the copies of the block in the current slot,
  // m1.. those of the next slots in ring order (the first n0 slots were
  // issued back to back)
  const int n0 = n_static < n_up ? n_static : n_up;
  int m0 = issued - (n0 - 1) * S::ops;
  int m1 = m0 + S::ops;
  int m2 = n0 > 2 ? m0 + 2 * S::ops : m1;
  int m3 = n0 > 3 ? m0 + 3 * S::ops : m1;
  int inflight = n0;
  int ramp = n0;   // next static block (and slot), two ahead of the current
  int off = 0;
  const int ring = depth * S::bytes;
  while (inflight > 0) {
    wait_slot<S::ops>(issued - m0);
    uint8_t* slot = slots + off;
    block_step<FAM, NA, BK, BV>(slot, lo, cst, ws);
    --inflight;
    int next = -1;
    if (cl.live) {
      const int v = claim_take<S::ops>(cl, lo.lane, issued - cl.mark);
      if (cl.base + v < cl.nblk) next = cl.base + v;
      else cl.live = false;
    }
    // every LDS read of this slot has returned before it is refilled
    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
    asm volatile("" ::: "memory");
    if (ramp < n_static) {
      issue_block<FAM, BK, BV>(g, blk0 + ramp * stride, lo.lane, slots + ramp * S::bytes);
      issued += S::ops;
      m2 = issued;
      ++ramp;
      ++inflight;
    }
    int mnew = m0;
    if (next >= 0) {
      claim_issue(cl.ctr, lo.lane);
      issued += 1;
      cl.mark = issued;
      issue_block<FAM, BK, BV>(g, next, lo.lane, slot);
      issued += S::ops;
      mnew = issued;
      ++inflight;
    }
    m0 = m1;
    m1 = depth == 2 ? mnew : m2;
    m2 = depth == 3 ? mnew : m3;
    m3 = mnew;
    off = off + S::bytes == ring ? 0 : off + S::bytes;
  }
}

// Dispatch on the unit's (K bits, V bits), uniform per workgroup; widths
// above MAXB are not instantiated.
template <int FAM, int NA, int MAXB>
__device__ __forceinline__ void dispatch(int bk, int bv, const Geo& g, int depth, int n_static,
                                         int n_up, int blk0, int stride, Claims& cl, int issued,
                                         uint8_t* slots, const LaneOps& lo, const uint32_t* cst,
                                         WaveState<NA>& ws) {
#define RQ_CASE(K, V)                                                              \
  case (K - 1) * 8 + (V - 1):                                                      \
    if (K <= MAXB && V <= MAXB)                                                    \
      stream_blocks<FAM, NA, (K <= MAXB ? K : 1), (V <= MAXB ? V : 1)>(            \
          g, depth, n_static, n_up, blk0, stride, cl, issued, slots, lo, cst, ws); \
    break;
#define RQ_ROW(K) RQ_CASE(K, 1) RQ_CASE(K, 2) RQ_CASE(K, 3) RQ_CASE(K, 4) \
                  RQ_CASE(K, 5) RQ_CASE(K, 6) RQ_CASE(K, 7) RQ_CASE(K, 8)
  switch ((bk - 1) * 8 + (bv - 1)) {
    RQ_ROW(1) RQ_ROW(2) RQ_ROW(3) RQ_ROW(4) RQ_ROW(5) RQ_ROW(6) RQ_ROW(7) RQ_ROW(8)
    default: break;
  }
#undef RQ_ROW
#undef RQ_CASE
}

// The 16-bit query rows of this kv-head as 16-byte pieces (thread tid holds
// piece tid: row tid / 16, channels 8 (tid % 16) ..), zero beyond G rows.
__device__ __forceinline__ u4 query_piece(const AttnLaunch& a, int b, int h) {
  const int tid = threadIdx.x;
  u4 v = {0u, 0u, 0u, 0u};
  if (tid < a.G * 16)
    v = reinterpret_cast<const u4*>(a.q + ((size_t)b * a.H * a.G + (size_t)h * a.G) * kD)[tid];
  return v;
}

// Copy the 16-bit query rows of this kv-head (G x 256 bytes) into qraw with
// buffer_load_dwordx4 .. lds: wave w moves bytes [1024 w, 1024 w + 1024).
// Returns the number of copy instructions this wave issued (0 or 1).
__device__ __forceinline__ int issue_query(const AttnLaunch& a, int b, int h, int wave,
                                           int lane, uint16_t* qraw) {
  const int bytes = a.G * kD * 2;
  if (1024 * wave >= bytes) return 0;
  const __amdgpu_buffer_rsrc_t src =
      buffer_of(a.q + ((size_t)b * a.H * a.G + (size_t)h * a.G) * kD, (uint32_t)bytes);
  if (1024 * wave + 16 * lane < bytes)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        src, (lds_void*)(reinterpret_cast<uint8_t*>(qraw) + 1024 * wave), 16,
        1024 * wave + 16 * lane, 0, 0, 0);
  return 1;
}

// Scaled query rows into qs (rows >= G zero), rotated for QuaRot.  Whole
// workgroup; piece from query_piece.
__device__ __forceinline__ void store_queries(const AttnLaunch& a, u4 piece, bool rotate,
                                              float (*qs)[kD]) {
  const int tid = threadIdx.x;
  float f = a.qscale;
  if (rotate) f *= kInvSqrtD;
  const float fs = rotate ? 1.0f : f;
  {
    const int j = tid >> 4, c = 8 * (tid & 15);
    const uint32_t w[4] = {piece.x, piece.y, piece.z, piece.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      qs[j][c + 2 * e] = widen(w[e] & 0xffffu, a.is_bf16) * fs;
      qs[j][c + 2 * e + 1] = widen(w[e] >> 16, a.is_bf16) * fs;
    }
  }
  __syncthreads();
  if (rotate) {
    for (int hh = 1; hh < kD; hh *= 2) {
      for (int e = tid; e < a.G * (kD / 2); e += kThreads) {
        const int j = e / (kD / 2), i = e % (kD / 2);
        const int base = (i / hh) * 2 * hh + (i % hh);
        const float x = qs[j][base], y = qs[j][base + hh];
        qs[j][base] = x + y;
        qs[j][base + hh] = x - y;
      }
      __syncthreads();
    }
    for (int e = tid; e < a.G * kD; e += kThreads) qs[e / kD][e % kD] *= f;
    __syncthreads();
  }
}

// TurboQuant: qs[j] = R q_j / sqrt(128) for the G query rows, on the
// matrix cores: D[row][coord] = Q . R^T with the 16-bit query rows (qraw,
// rows >= G unused) as A and rows of R (global memory, bf16; converted to
// fp16 for fp16 queries) as B.  Wave w computes coordinate tiles 2w, 2w+1.
typedef __bf16 abf8 __attribute__((ext_vector_type(8)));

// What the TurboQuant set-up reads from global memory, loaded before the
// query and the first block copies (so that waiting for it never waits
// for a copy): this lane's B operands of the query rotation (rows of R)
// and the codebook entries of its LDS table entries.
struct TurboPrefetch {
  u4 rb[2][4];      // [tile t][k-step]: R row 16 (2 wave + t) + r, 8 entries
  float c[2][2];    // [side][lo, hi]: centroids of table entry tid of the side
};

__device__ __forceinline__ void turbo_prefetch(const AttnLaunch& a, int h, int bk, int bv,
                                               TurboPrefetch& p) {
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid & (kWave - 1);
  const int r = lane & 15, g = lane >> 4;
  const RQ_GLOBAL u4* Rh = gptr(reinterpret_cast<const u4*>(a.rot + (size_t)h * kD * kD));
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      p.rb[t][ks] = Rh[((16 * (2 * wave + t) + r) * kD + 32 * ks + 8 * g) / 8];
  // table entry k = tid of each side: centroid k (widths >= 5) or the pair
  // (k mod 2^b, k / 2^b) (widths 2..4); indices < 256 stay inside the
  // width's 512-entry row of the codebook table
#pragma unroll
  for (int side = 0; side < 2; ++side) {
    const int bb = side ? bv : bk;
    const RQ_GLOBAL float* c = gptr(a.cb + (bb - 1) * 512 + 256);
    p.c[side][0] = c[bb >= 5 ? tid : (tid & ((1 << bb) - 1))];
    p.c[side][1] = c[(tid >> bb) & 255];
  }
}

__device__ __forceinline__ void rotate_queries(const AttnLaunch& a, const TurboPrefetch& p,
                                               const uint16_t* qraw, float (*qs)[kD]) {
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid & (kWave - 1);
  const int r = lane & 15, g = lane >> 4;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int nt = 2 * wave + t;
    f4 d = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      // rows >= G (outputs unused) read row 0: qraw holds G rows
      const u4 qa = *reinterpret_cast<const u4*>(&qraw[(r < a.G ? r : 0) * kD + 32 * ks + 8 * g]);
      u4 rb = p.rb[t][ks];
      if (a.is_bf16) {
        d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(abf8, qa),
                                                    __builtin_bit_cast(abf8, rb), d, 0, 0, 0);
      } else {
        uint32_t w[4] = {rb.x, rb.y, rb.z, rb.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const _Float16 lo = (_Float16)__uint_as_float(w[e] << 16);
          const _Float16 hi = (_Float16)__uint_as_float(w[e] & 0xffff0000u);
          w[e] = (uint32_t)__builtin_bit_cast(uint16_t, lo) |
                 ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
        }
        rb = (u4){w[0], w[1], w[2], w[3]};
        d = mfma(u4_h8(qa), u4_h8(rb), d);
      }
    }
    // lane: coordinate 16 nt + r of query rows 4g .. 4g+3
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = 4 * g + i;
      if (j < a.G) qs[j][16 * nt + r] = d[i] * kInvSqrtD;
    }
  }
  __syncthreads();
}

// Partial of (unit, slot): float [G][2 + 128] = (max, sum, acc[128]).
// Slots of a unit: 0 .. nw-1 streaming, nw .. nw+n_rw-1 the window,
// then the group partials of the two-level merge.
__device__ __forceinline__ float* part_ptr(const AttnLaunch& a, size_t unit, int slot) {
  return a.part + (unit * a.pstride + slot) * (size_t)a.G * (2 + kD);
}

// Residual-window staging: 64 tokens of K and of V per chunk, rows padded
// to 272 bytes so that lanes reading different rows spread over the banks.
constexpr int kResTok = 64;
constexpr int kResRow = 136;   // uint16 per padded row
constexpr size_t kResLds = (size_t)2 * kResTok * kResRow * sizeof(uint16_t);

// Tokens t_lo .. t_hi-1 of the 16-bit residual window of one unit, original
// domain.  They are read in chunks of 64 tokens staged in LDS; the loads of the next chunk (and of
// the queries, before the first) are in flight while a chunk is computed.
// Wave w takes query rows w, w+4, ...; lane = token for the scores, lane =
// channel pair for PV.  stage: LDS for one chunk (kResLds bytes), qs: LDS
// for the query rows.
template <bool BF16>
__device__ __forceinline__ void residual_slot_t(const AttnLaunch& a, int b, int h,
                                                float (*qs)[kD], uint16_t* stage,
                                                float* dst, int t_lo, int t_hi) {
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid & (kWave - 1);
  const int cap = a.R + kChunk;
  const uint16_t* kb = a.resid + (((size_t)b * a.H + h) * 2 + 0) * cap * kD;
  const uint16_t* vb = a.resid + (((size_t)b * a.H + h) * 2 + 1) * cap * kD;
  // a token appended by this call is read from the new input (its window
  // slot is written below, by the one workgroup whose range holds it)
  const size_t unit_row = ((size_t)b * a.H + h) * kD;
  const uint16_t* kn = a.t_new >= 0 ? a.k_new + unit_row : kb;
  const uint16_t* vn = a.t_new >= 0 ? a.v_new + unit_row : vb;
  uint16_t* ks = stage;
  uint16_t* vs = stage + kResTok * kResRow;
  // a chunk is 64 tokens x 16 pieces of 16 bytes: four pieces per thread
  u4 kr[4], vr[4];
  auto load_chunk = [&](int t0) {
    const int n = (t_hi - t0) < kResTok ? (t_hi - t0) : kResTok;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = tid + i * kThreads, t = e >> 4, piece = e & 15;
      if (t < n) {
        const bool fresh = t0 + t == a.t_new;
        const size_t row = fresh ? (size_t)piece * 8 : (size_t)((t0 + t) % cap) * kD + piece * 8;
        kr[i] = *reinterpret_cast<const u4*>((fresh ? kn : kb) + row);
        vr[i] = *reinterpret_cast<const u4*>((fresh ? vn : vb) + row);
      }
    }
  };
  const u4 qpiece = query_piece(a, b, h);
  if (t_lo < t_hi) load_chunk(t_lo);
  store_queries(a, qpiece, false, qs);
  float m_run[4], l_run[4], ac0[4], ac1[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    m_run[q] = -INFINITY;
    l_run[q] = 0.0f;
    ac0[q] = 0.0f;
    ac1[q] = 0.0f;
  }
  for (int t0 = t_lo; t0 < t_hi; t0 += kResTok) {
    const int n = (t_hi - t0) < kResTok ? (t_hi - t0) : kResTok;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = tid + i * kThreads, t = e >> 4, piece = e & 15;
      if (t < n) {
        *reinterpret_cast<u4*>(ks + t * kResRow + piece * 8) = kr[i];
        *reinterpret_cast<u4*>(vs + t * kResRow + piece * 8) = vr[i];
        if (t0 + t == a.t_new) {
          uint16_t* w = a.resid_w + (size_t)(a.t_new % cap) * kD + piece * 8;
          *reinterpret_cast<u4*>(w + (((size_t)b * a.H + h) * 2 + 0) * cap * kD) = kr[i];
          *reinterpret_cast<u4*>(w + (((size_t)b * a.H + h) * 2 + 1) * cap * kD) = vr[i];
        }
      }
    }
    __syncthreads();
    if (t0 + kResTok < t_hi) load_chunk(t0 + kResTok);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = wave + kWaves * q;
      if (j >= a.G) break;
      float s = -INFINITY;
      if (lane < n) {
        s = 0.0f;
        const u4* krow = reinterpret_cast<const u4*>(ks + lane * kResRow);
#pragma unroll 4
        for (int c8 = 0; c8 < kD / 8; ++c8) {
          const u4 w = krow[c8];
          const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            s = __builtin_fmaf(qs[j][8 * c8 + 2 * e], widen_t<BF16>(ww[e] & 0xffffu), s);
            s = __builtin_fmaf(qs[j][8 * c8 + 2 * e + 1], widen_t<BF16>(ww[e] >> 16), s);
          }
        }
      }
      float mx = s;
      for (int d = 32; d >= 1; d >>= 1) mx = __builtin_fmaxf(mx, xor_shfl(mx, d));
      const float mn = __builtin_fmaxf(m_run[q], mx);
      const float al = __builtin_amdgcn_exp2f(m_run[q] - mn);
      const float p = lane < n ? __builtin_amdgcn_exp2f(s - mn) : 0.0f;
      float sum = p;
      for (int d = 32; d >= 1; d >>= 1) sum += xor_shfl(sum, d);
      l_run[q] = l_run[q] * al + sum;
      m_run[q] = mn;
      float c0 = ac0[q] * al, c1 = ac1[q] * al;
#pragma unroll 8
      for (int i = 0; i < n; ++i) {
        const uint32_t w = *reinterpret_cast<const uint32_t*>(vs + i * kResRow + 2 * lane);
        const float pi = __builtin_bit_cast(
            float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, p), i));
        c0 = __builtin_fmaf(pi, widen_t<BF16>(w & 0xffffu), c0);
        c1 = __builtin_fmaf(pi, widen_t<BF16>(w >> 16), c1);
      }
      ac0[q] = c0;
      ac1[q] = c1;
    }
    __syncthreads();
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int j = wave + kWaves * q;
    if (j >= a.G) break;
    float* d = dst + (size_t)j * (2 + kD);
    if (lane == 0) {
      st_agent(d, m_run[q]);
      st_agent(d + 1, l_run[q]);
    }
    st_agent(d + 2 + 2 * lane, ac0[q]);
    st_agent(d + 2 + 2 * lane + 1, ac1[q]);
  }
}

__device__ __forceinline__ void residual_slot(const AttnLaunch& a, int b, int h,
                                              float (*qs)[kD], uint16_t* stage,
                                              float* dst, int t_lo, int t_hi) {
  if (a.is_bf16) residual_slot_t<true>(a, b, h, qs, stage, dst, t_lo, t_hi);
  else residual_slot_t<false>(a, b, h, qs, stage, dst, t_lo, t_hi);
}

// Quantized blocks of workgroup slot `slot` of unit (b, h): stream, merge the
// four waves and write the slot's partial.
template <int FAM, int NA, int MAXB>
__device__ __forceinline__ void stream_slot(const AttnLaunch& a, int slot, int nw, int h, int b,
                                            float (*qs)[kD], uint16_t* qraw, uint32_t* cst,
                                            uint8_t* slots, float* merge) {
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid & (kWave - 1);
  const size_t unit = (size_t)b * a.H + h;
  const int G = a.G;
  const int bk = kernarg_byte(&a.tab.bits[0][0], 2 * h),
            bv = kernarg_byte(&a.tab.bits[0][0], 2 * h + 1);
  const int nblk_cap = a.cap / kChunk;
  constexpr int mk = meta_block_bytes(FAM, 0), mv = meta_block_bytes(FAM, 1);
  Geo g;
  {
    // the unit's codes and metadata as two byte ranges (the host checks
    // that each spans less than 4 GiB)
    const size_t k0 = a.tab.code_off[h][0] + (size_t)b * a.cap * 16 * bk;
    const size_t v0 = a.tab.code_off[h][1] + (size_t)b * a.cap * 16 * bv;
    const size_t km0 = meta_unit_offset(FAM, h, 0, b, a.B, nblk_cap);
    const size_t vm0 = meta_unit_offset(FAM, h, 1, b, a.B, nblk_cap);
    g.voff = (uint32_t)(v0 - k0);
    g.vmoff = (uint32_t)(vm0 - km0);
    g.codes = buffer_of(a.codes + k0, g.voff + (uint32_t)a.cap * 16 * bv);
    g.meta = buffer_of(a.meta + km0, g.vmoff + (uint32_t)nblk_cap * mv);
  }
  const int nblk = a.nq / kChunk;
  // this unit's ring: as many whole blocks as the wave's region holds
  const int blk_bytes = 512 * (bk + bv) + mk + mv;
  int depth = a.wave_bytes / blk_bytes;
  depth = depth < kMaxDepth ? depth : kMaxDepth;
  uint8_t* my_slots = slots + (size_t)wave * a.wave_bytes;
  // The unit's blocks are split between its claim groups (kGroup
  // workgroups each) in proportion to their sizes.  Inside a group the
  // first `depth` blocks of every wave are assigned statically (wave k of
  // the group's 4 n waves: blocks lo + k, lo + k + 4 n, ...) and the rest
  // are claimed from the group's counter.  Query copy first, then the first
  // claim and the first block: waiting for the queries leaves those in
  // flight.  The second block follows once the query operands are built,
  // the others while the first ones are computed.
  const int grp = slot / kGroup;
  const int gw0 = grp * kGroup;
  const int gn = nw - gw0 < kGroup ? nw - gw0 : kGroup;
  const int g_lo = (int)((long)nblk * gw0 / nw);
  const int g_hi = (int)((long)nblk * (gw0 + gn) / nw);
  const int wk = (slot - gw0) * kWaves + wave, wstride = gn * kWaves;
  int n_static = 0;
  for (int j = 0; j < depth; ++j) n_static += g_lo + wk + j * wstride < g_hi ? 1 : 0;
  Claims cl;
  cl.ctr = a.counters + unit * a.cstride + a.claim_off + 16 * grp;
  cl.epoch = a.epoch;
  cl.base = g_lo + depth * wstride;
  cl.nblk = g_hi;
  cl.live = cl.base < g_hi;
  cl.mark = 0;
  TurboPrefetch tp;
  if (FAM == RQ_TURBO) turbo_prefetch(a, h, bk, bv, tp);
  const int nq_ops = issue_query(a, b, h, wave, lane, qraw);
  int issued = 0;
  if (cl.live) {
    claim_issue(cl.ctr, lane);
    issued += 1;
    cl.mark = issued;
  }
  const int nb_ops = issue_first(g, bk, bv, mk, mv, 0, 1, g_lo + wk, wstride, g_hi, lane,
                                 my_slots);
  if (nq_ops) wait_vm_rt(issued + nb_ops);
  issued += nb_ops;
  if (tid < 8) cst[tid] = tid < 4 ? kOnes : 0u;
  __syncthreads();
  LaneOps lo;
  lo.lane = lane;
  lo.r = lane >> 4;
  lo.col = lane & 15;
  lo.GP = a.GP;
  lo.gsub = lo.col / a.GP;
  lo.tabk = lo.tabv = nullptr;
  {
    // this lane's query row j = col mod GP, channels 32 r .. 32 r + 31
    // (the rotated row for QuaRot and TurboQuant), scaled
    const int j = lo.col & (a.GP - 1);
    float qv[32];
    if (FAM == RQ_TURBO) {
      // LDS tables of the unit's K and V widths (pairs for 2..4 bits,
      // centroids above); rotate_queries ends with a barrier
      uint8_t* tab = reinterpret_cast<uint8_t*>(qs) + (size_t)G * kD * sizeof(float);
      static_assert(kThreads == 256, "one table entry of each side per thread");
#pragma unroll
      for (int side = 0; side < 2; ++side) {
        const int k = tid, bb = side ? bv : bk;
        uint8_t* area = tab + side * kTqTabBytes;
        if (bb >= 5) {
          if (k < (1 << bb)) reinterpret_cast<_Float16*>(area)[k] = (_Float16)tp.c[side][0];
        } else if (bb >= 2 && k < (1 << (2 * bb))) {
          const h2 v = {(_Float16)tp.c[side][0], (_Float16)tp.c[side][1]};
          reinterpret_cast<uint32_t*>(area)[k] = as_u32(v);
        }
      }
      lo.tabk = (lds_h*)tab;
      lo.tabv = (lds_h*)(tab + kTqTabBytes);
      rotate_queries(a, tp, qraw, qs);
#pragma unroll
      for (int i = 0; i < 32; ++i) qv[i] = j < G ? qs[j][32 * lo.r + i] : 0.0f;
    } else {
      const u4* src = reinterpret_cast<const u4*>(qraw + j * kD + 32 * lo.r);
#pragma unroll
      for (int c8 = 0; c8 < 4; ++c8) {
        const u4 w4 = j < G ? src[c8] : (u4){0u, 0u, 0u, 0u};
        const uint32_t w[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          qv[8 * c8 + 2 * e] = widen(w[e] & 0xffffu, a.is_bf16);
          qv[8 * c8 + 2 * e + 1] = widen(w[e] >> 16, a.is_bf16);
        }
      }
      // RTN runs this instantiation with codes in the original domain
      if (FAM == RQ_QUAROT && a.family == RQ_QUAROT) {
        // unnormalised Walsh-Hadamard transform of the row, stages of
        // stride 1, 2, .., 64 (lower index x + y, upper x - y): strides up
        // to 16 inside the lane's 32 channels, 32 and 64 across the lanes
        // holding the other quarters (r ^ 1, r ^ 2)
#pragma unroll
        for (int hh = 1; hh < 32; hh *= 2)
#pragma unroll
          for (int i = 0; i < 32; ++i)
            if ((i & hh) == 0) {
              const float x = qv[i], y = qv[i + hh];
              qv[i] = x + y;
              qv[i + hh] = x - y;
            }
#pragma unroll
        for (int st = 1; st <= 2; st *= 2) {
          const bool upper = (lo.r & st) != 0;
#pragma unroll
          for (int i = 0; i < 32; ++i) {
            const float o = xor_shfl(qv[i], 16 * st);
            qv[i] = upper ? o - qv[i] : qv[i] + o;
          }
        }
#pragma unroll
        for (int i = 0; i < 32; ++i) qv[i] *= kInvSqrtD;
      }
    }
    // row exponent e: the row's largest |q'| is below 2^e (frexp), so every
    // q' 2^-e lies in (-1, 1); 0 for a zero row.  The softmax scale
    // (scale * log2 e) is applied to the fp32 scores, so the operands of
    // unrotated queries are the 16-bit inputs times powers of two, exact.
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < 32; ++i) amax = __builtin_fmaxf(amax, __builtin_fabsf(qv[i]));
    amax = __builtin_fmaxf(amax, xor_shfl(amax, 16));
    amax = __builtin_fmaxf(amax, xor_shfl(amax, 32));
    const int e = amax > 0.0f ? __builtin_amdgcn_frexp_expf(amax) : 0;
    lo.cK = __builtin_ldexpf(a.qscale, FAM == RQ_TURBO ? e : 24 + e);
    lo.eK = __builtin_ldexpf(a.qscale, e);
    // static QK operands: k-slot pair (kb, k') = channels 32r + 4kb + k'
    // and 32r + 16 + 4kb + k'
    const int8_t* kp = a.fpos.k[bk];
    const int8_t* vp = a.fpos.v[bv];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const float q0 = qv[4 * kb + kk], q1 = qv[16 + 4 * kb + kk];
        const int sh = FAM == RQ_TURBO ? -e : -e - kp[4 * kb + kk];
        const h2 vh = {(_Float16)__builtin_ldexpf(q0, sh), (_Float16)__builtin_ldexpf(q1, sh)};
        const h2 vz = {(_Float16)__builtin_ldexpf(q0, -e), (_Float16)__builtin_ldexpf(q1, -e)};
        lo.qh[4 * kb + kk] = as_u32(vh);
        lo.qz[4 * kb + kk] = as_u32(vz);
      }
#pragma unroll
    for (int i = 0; i < 4; ++i) lo.vq[i] = h_pair((uint32_t)(15 + vp[i]) << 10);
    lo.corrK = (f4){0.f, 0.f, 0.f, 0.f};
    if (FAM == RQ_TURBO) {
      lo.lut1 = tq_make_lut1(a.cb);
    }
    if (key_fam(FAM) == RQ_QUAROT) {
      // the symmetric offset of the key codes, -2^(b-1) at the codes'
      // weights 2^(kpos-24) (exact subnormals), against the query operands
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        uint32_t c[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          c[kk] = h_pair(0x8000u | (1u << (bk - 1 + kp[4 * kb + kk])));
        lo.corrK = mfma(make_h8(c[0], c[1], c[2], c[3]),
                        make_h8(lo.qh[4 * kb], lo.qh[4 * kb + 1], lo.qh[4 * kb + 2],
                                lo.qh[4 * kb + 3]),
                        lo.corrK);
      }
    }
  }
  // the rest of the ring, now that the set-up is done
  issued += issue_first(g, bk, bv, mk, mv, 1, depth, g_lo + wk, wstride, g_hi, lane, my_slots);
  WaveState<NA> ws;
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) ws.acc[nt] = (f4){0.f, 0.f, 0.f, 0.f};
  ws.corrO = (f4){0.f, 0.f, 0.f, 0.f};
  ws.corrZ = (f4){0.f, 0.f, 0.f, 0.f};
  ws.m_run = -INFINITY;
  ws.ev = 0;
  {
    // value slots' 2^-vpos (TurboQuant: 1), the exponent Ev = 0
    const int8_t* vp = a.fpos.v[bv];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      ws.wv[i] = h_pair((uint32_t)(15 - (FAM == RQ_TURBO ? 0 : vp[i])) << 10);
  }

  // blocks at normal priority; what comes before and after at raised
  // priority (see attn_kernel)
  __builtin_amdgcn_s_setprio(0);
  dispatch<FAM, NA, MAXB>(bk, bv, g, depth, n_static, depth, g_lo + wk, wstride, cl, issued,
                          my_slots, lo, cst, ws);
  __builtin_amdgcn_s_setprio(kSetupPrio);

  // ---- this wave's result per query row: (m, l, out[128]) in canonical form
  const int r = lo.r, col = lo.col, GP = a.GP;
  constexpr int GPA = 4 / NA;
  float zt[4][4], lrow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int gg = 0; gg < 4; ++gg) zt[gg][i] = __shfl(ws.corrZ[i], r * 16 + gg, kWave);
    lrow[i] = __shfl(ws.corrZ[i], r * 16 + (val_fam(FAM) == RQ_KIVI ? 4 : 0), kWave);
  }
  float mrow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) mrow[i] = __shfl(ws.m_run, (4 * r + i) & (GP - 1), kWave);
  // scale of the value sums: 2^(24+Ev) for codes as subnormals (QuaRot and
  // RTN: 2^Ev times 2^24 acc minus the offset 2^(b-1) corrO), 2^Ev / sqrt(128)
  // for TurboQuant
  constexpr int VF = val_fam(FAM);
  const float cv = VF == RQ_TURBO ? __builtin_ldexpf(kInvSqrtD, ws.ev)
                                  : __builtin_ldexpf(1.0f, VF == RQ_QUAROT ? ws.ev : 24 + ws.ev);
  const float voff = (float)(1 << (bv - 1));
  __syncthreads();   // every wave is done with its slot
  float* mw = merge + (size_t)wave * G * (2 + kD);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * r + i, jj = row & (GP - 1), gs = row / GP;
    if (jj < G) {
      if (VF == RQ_KIVI) {
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) {
          const int gt = nt / 2;
          if (gs == gt % GPA)
            mw[jj * (2 + kD) + 2 + 16 * nt + col] = __builtin_fmaf(ws.acc[nt][i], cv, zt[gt][i]);
        }
        if (gs == 0 && col == 0) {
          mw[jj * (2 + kD)] = mrow[i];
          mw[jj * (2 + kD) + 1] = lrow[i];
        }
      } else if (gs == 0) {
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) {
          float v;
          if (VF == RQ_QUAROT)
            v = __builtin_fmaf(ws.acc[nt][i], 16777216.0f, -voff * ws.corrO[i]) * cv;
          else
            v = ws.acc[nt][i] * cv;
          mw[jj * (2 + kD) + 2 + 16 * nt + col] = v;
        }
        if (col == 0) {
          mw[jj * (2 + kD)] = mrow[i];
          mw[jj * (2 + kD) + 1] = lrow[i];
        }
      }
    }
  }
  __syncthreads();
  float* dst = part_ptr(a, unit, slot);
  for (int e = tid; e < G * kD; e += kThreads) {
    const int j = e / kD, cc = e % kD;
    float M = -INFINITY;
    for (int w = 0; w < kWaves; ++w) M = __builtin_fmaxf(M, merge[(w * G + j) * (2 + kD)]);
    float acc = 0.0f, l = 0.0f;
    for (int w = 0; w < kWaves; ++w) {
      const float* src = merge + (size_t)(w * G + j) * (2 + kD);
      const float f = (src[0] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(src[0] - M);
      acc = __builtin_fmaf(f, src[2 + cc], acc);
      l = __builtin_fmaf(f, src[1], l);
    }
    st_agent(dst + j * (2 + kD) + 2 + cc, acc);
    if (cc == 0) {
      st_agent(dst + j * (2 + kD), M);
      st_agent(dst + j * (2 + kD) + 1, l);
    }
  }
}

// Merge partials of one (batch, kv-head) unit: slots first .. first+count-1
// (quantized blocks: QuaRot and TurboQuant in the rotated domain) and the
// nwin window slots win .. win+nwin-1 (original domain).  dst: a partial
// slot to write the merged (max, sum, acc) to, or NULL to write the unit's
// output.  Thread t owns E consecutive elements of one query row (E = 128 Gp
// / 256, Gp the power of two >= G), so a slot's (max, sum) is loaded once
// per row segment; the loads of several slots are in flight together.
// Whole workgroup; lds: scratch of 128 G floats, plus the rotation
// (TurboQuant, 32 KB).
template <int E>
__device__ __forceinline__ void merge_rows(const AttnLaunch& a, size_t unit, float* lds,
                                           int first, int count, int win, int nwin,
                                           float* dst) {
  constexpr int kS = E <= 2 ? 16 : (E == 4 ? 12 : 6);
  constexpr int TPR = kD / E;              // threads per row
  const int tid = threadIdx.x;
  const int G = a.G;
  const int j = tid / TPR, c0 = (tid % TPR) * E;
  const bool own = j < G;
  const int ns = count + nwin;
  const float* base = part_ptr(a, unit, 0) + (size_t)j * (2 + kD);
  const size_t stride = (size_t)G * (2 + kD);
  // TurboQuant output: the unit's rotation (32 KB) is loaded now, in flight
  // with the partials, and staged in LDS after them
  constexpr int kRotLoads = kD * kD / 8 / kThreads;
  const bool turbo_out = !dst && a.family == RQ_TURBO;
  u4 rtmp[kRotLoads];
  if (turbo_out) {
    const RQ_GLOBAL u4* src = gptr(reinterpret_cast<const u4*>(
        a.rot + (size_t)(unit % a.H) * kD * kD));
#pragma unroll
    for (int k = 0; k < kRotLoads; ++k) rtmp[k] = src[tid + k * kThreads];
  }
  float M = -INFINITY, den = 0.0f, num[E], tail[E];
#pragma unroll
  for (int k = 0; k < E; ++k) num[k] = tail[k] = 0.0f;
  if (own) {
    for (int s0 = 0; s0 < ns; s0 += kS) {
      float m[kS], l[kS], v[kS][E];
#pragma unroll
      for (int i = 0; i < kS; ++i) {
        m[i] = -INFINITY;
        l[i] = 0.0f;
#pragma unroll
        for (int k = 0; k < E; ++k) v[i][k] = 0.0f;
        if (s0 + i < ns) {
          const int slot = s0 + i < count ? first + s0 + i : win + (s0 + i - count);
          const float* src = base + slot * stride;
          m[i] = ld_agent(src);
          l[i] = ld_agent(src + 1);
#pragma unroll
          for (int k = 0; k < E; ++k) v[i][k] = ld_agent(src + 2 + c0 + k);
        }
      }
#pragma unroll
      for (int i = 0; i < kS; ++i) {
        if (!(l[i] > 0.0f)) continue;
        const float mn = __builtin_fmaxf(M, m[i]);
        const float fo = __builtin_amdgcn_exp2f(M - mn);
        const float fi = __builtin_amdgcn_exp2f(m[i] - mn);
        M = mn;
        den = __builtin_fmaf(den, fo, fi * l[i]);
        // the window slot is in the original domain: kept apart
        const bool w = s0 + i >= count;
#pragma unroll
        for (int k = 0; k < E; ++k) {
          num[k] = num[k] * fo + (w ? 0.0f : fi * v[i][k]);
          tail[k] = tail[k] * fo + (w ? fi * v[i][k] : 0.0f);
        }
      }
    }
  }
  if (dst) {
    // a group partial (no window in it)
    if (own) {
      float* d = dst + (size_t)j * (2 + kD);
      if (c0 == 0) {
        st_agent(d, M);
        st_agent(d + 1, den);
      }
#pragma unroll
      for (int k = 0; k < E; ++k) st_agent(d + 2 + c0 + k, num[k]);
    }
    return;
  }
  float* out = a.out + unit * G * kD + (size_t)j * kD + c0;   // (b, h) -> rows h*G..
  const float inv = own ? 1.0f / den : 0.0f;
  if (a.family == RQ_KIVI || a.family == RQ_RTN || a.family == RQ_KIVI_RTN) {
    if (own)
#pragma unroll
      for (int k = 0; k < E; ++k) out[k] = (num[k] + tail[k]) * inv;
    return;
  }
  float* rot = lds;                        // [G][128] quantized-domain sums
  if (own)
#pragma unroll
    for (int k = 0; k < E; ++k) rot[j * kD + c0 + k] = num[k];
  if (a.family == RQ_QUAROT) {
    // x = H y / sqrt(128)
    __syncthreads();
    for (int hh = 1; hh < kD; hh *= 2) {
      for (int e = tid; e < G * (kD / 2); e += kThreads) {
        const int jj = e / (kD / 2), i = e % (kD / 2);
        const int bse = (i / hh) * 2 * hh + (i % hh);
        const float x = rot[jj * kD + bse], y = rot[jj * kD + bse + hh];
        rot[jj * kD + bse] = x + y;
        rot[jj * kD + bse + hh] = x - y;
      }
      __syncthreads();
    }
    if (own)
#pragma unroll
      for (int k = 0; k < E; ++k)
        out[k] = rot[j * kD + c0 + k] * kInvSqrtD * inv + tail[k] * inv;
    return;
  }
  // TurboQuant: x = R^T y, R staged in LDS (row-major, as stored)
  uint16_t* Rs = reinterpret_cast<uint16_t*>(lds + G * kD);
#pragma unroll
  for (int k = 0; k < kRotLoads; ++k) reinterpret_cast<u4*>(Rs)[tid + k * kThreads] = rtmp[k];
  __syncthreads();
  if (own) {
    float acc[E];
#pragma unroll
    for (int k = 0; k < E; ++k) acc[k] = 0.0f;
    for (int cp = 0; cp < kD; ++cp) {
      const float y = rot[j * kD + cp];
#pragma unroll
      for (int k = 0; k < E; ++k)
        acc[k] = __builtin_fmaf(__uint_as_float((uint32_t)Rs[cp * kD + c0 + k] << 16), y, acc[k]);
    }
#pragma unroll
    for (int k = 0; k < E; ++k) out[k] = acc[k] * inv + tail[k] * inv;
  }
}

__device__ __forceinline__ void merge_slots(const AttnLaunch& a, size_t unit, float* lds,
                                            int first, int count, int win, int nwin,
                                            float* dst) {
  if (a.GP <= 2)
    merge_rows<1>(a, unit, lds, first, count, win, nwin, dst);
  else if (a.GP <= 4)
    merge_rows<2>(a, unit, lds, first, count, win, nwin, dst);
  else if (a.GP <= 8)
    merge_rows<4>(a, unit, lds, first, count, win, nwin, dst);
  else
    merge_rows<8>(a, unit, lds, first, count, win, nwin, dst);
}

// Arrival tickets on the unit's counters (agent scope); the caller's
// partials are published (s_waitcnt 0) before.
__device__ __forceinline__ uint32_t take_ticket(uint64_t* counter, uint32_t epoch) {
  __shared__ uint32_t ticket;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) ticket = ctr_count(counter, ctr_add(counter), epoch);
  __syncthreads();
  return ticket;
}

// A counter's last use in the call: ready it for the next call.
__device__ __forceinline__ void reset_counter(uint64_t* counter, uint32_t epoch) {
  if (threadIdx.x == 0)
    __hip_atomic_store(counter, (uint64_t)next_epoch(epoch) << 32, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

// FAM: quantizer family; NA: A operands of the KIVI value side (G <= 4: 1,
// G <= 8: 2, else 4); MAXB: largest bit-width handled (4 or 8).
// The compiler allocates v0..v165 (the attribute's value is doubled for the
// unified vector register file of this architecture: 83 -> 166);
// v[166:167], the rest of the 168 that three workgroups per CU leave a
// lane, hold the block claims.
template <int FAM, int NA, int MAXB>
__global__ void __launch_bounds__(kThreads, kAttnOcc) __attribute__((amdgpu_num_vgpr(83)))
attn_kernel(AttnLaunch a) {
  __shared__ u4 cst4[2];             // fp16 ones (4 dwords), zeros (4 dwords)
  uint32_t* cst = reinterpret_cast<uint32_t*>(cst4);
  // one area used in turn for the waves' block rings while streaming and
  // the wave merge area [kWaves][G][2 + 128] floats (window workgroups:
  // staging, then their scaled query rows); behind it the G 16-bit query
  // rows (uint16 [G][128]) and, for TurboQuant, the G rotated rows (float
  // [G][128])
  extern __shared__ u4 dyn[];
  uint8_t* slots = reinterpret_cast<uint8_t*>(dyn);
  float* merge = reinterpret_cast<float*>(dyn);
  uint16_t* qraw = reinterpret_cast<uint16_t*>(slots + a.area_bytes);
  float (*qs)[kD] = reinterpret_cast<float (*)[kD]>(slots + a.area_bytes + a.G * kD * 2);
  // Flat grid, unit index fastest and skewed by one per slot: the nw
  // workgroups of a unit are about n_units apart in dispatch order, so they
  // land in every residency round of the CUs (the workgroups sharing a CU
  // issue at different rates, the older first), and on different XCDs
  // (workgroups go to the XCDs round-robin).  Block claims then balance
  // each unit over fast and slow slots alike.
  const int n_units = a.B * a.H;
  const int slot = blockIdx.x / n_units;
  const size_t unit = (blockIdx.x + slot) % n_units;
  const int h = (int)(unit % a.H), b = (int)(unit / a.H);
  // this unit's workgroups (its kv-head's share of the grid; slots beyond
  // it have nothing to do)
  const int nw = a.nwg[h];
  const int nx = nw > 0 ? nw : 1;
  if (slot >= nx) return;
  // Set-up, the window, the partial write and the merges run at a raised
  // wave priority: they share SIMDs with other workgroups' block loops, and
  // a unit finishes only after its slowest set-up and its merge, so they
  // go first; the block loops run at normal priority.
  __builtin_amdgcn_s_setprio(kSetupPrio);
  // The unit's nx workgroups: slot s first takes the 16-bit window chunks
  // s, s + nx, .. (kResChunk tokens each, partial nw + chunk; the area is
  // their staging), then streams its share of the quantized blocks (slots
  // 0 .. nw-1).  The window thus costs a few workgroups some of their
  // blocks (the claims hand those to the others) instead of holding
  // workgroups of its own.
  for (int c = slot; c < a.n_rw; c += nx) {
    const int t_lo = a.nq + c * kResChunk;
    const int t_hi = t_lo + kResChunk < a.n_tokens ? t_lo + kResChunk : a.n_tokens;
    residual_slot(a, b, h, reinterpret_cast<float (*)[kD]>(slots + kResLds),
                  reinterpret_cast<uint16_t*>(slots), part_ptr(a, unit, nw + c), t_lo, t_hi);
    __syncthreads();   // the staging area is reused
  }
  // the block stream counts this wave's memory operations from zero: the
  // window's partial stores complete first
  if (slot < a.n_rw) wait_vm<0>();
  if (slot < nw) stream_slot<FAM, NA, MAXB>(a, slot, nw, h, b, qs, qraw, cst, slots, merge);
  // publish this workgroup's partials and take a ticket.  Up to
  // kAttnMergeFlat workgroups: the last to arrive merges every slot and the
  // window.  More: they report in groups of kGroup, the last of a group
  // merges it into a group partial; the group mergers then report on the
  // final counter, whose last arrival merges the group partials and the
  // window.  Every counter used is left ready for the next call.
  uint64_t* cnt = a.counters + unit * a.cstride;
  const uint32_t ep = a.epoch;
  const int ng = (nw + kGroup - 1) / kGroup;
  if (nw <= kAttnMergeFlat) {
    if (take_ticket(cnt, ep) == (uint32_t)(nx - 1)) {
      merge_slots(a, unit, merge, 0, nw, nw, a.n_rw, nullptr);
      reset_counter(cnt, ep);
      // every claim group's line (the last arrival: nobody claims now)
      for (int g = 0; g < (ng > 1 ? ng : 1); ++g) reset_counter(cnt + a.claim_off + 16 * g, ep);
    }
    return;
  }
  {
    // two levels: every workgroup streams (nx = nw > kAttnMergeFlat)
    const int g = slot / kGroup;
    const int gsz = nw - g * kGroup < kGroup ? nw - g * kGroup : kGroup;
    if (take_ticket(cnt + 1 + g, ep) != (uint32_t)(gsz - 1)) return;
    __syncthreads();   // the merge area is read until here
    merge_slots(a, unit, merge, g * kGroup, gsz, 0, 0,
                part_ptr(a, unit, nw + a.n_rw + g));
    reset_counter(cnt + 1 + g, ep);
    // every wave of the group has stopped claiming
    reset_counter(cnt + a.claim_off + 16 * g, ep);
  }
  if (take_ticket(cnt, ep) != (uint32_t)(ng - 1)) return;
  merge_slots(a, unit, merge, nw + a.n_rw, ng, nw, a.n_rw, nullptr);
  reset_counter(cnt, ep);
}

}  // namespace

}  // namespace rq

// Defines hipError_t NAME(const AttnLaunch&, size_t lds, hipStream_t):
// launches attn_kernel<FAM, NA, MAXB> over the unit grid.
#define RQ_DEFINE_ATTN_LAUNCHER(FAM, NA, MAXB, NAME)                            \
  namespace rq {                                                                \
  hipError_t NAME(const AttnLaunch& a, size_t lds, hipStream_t s) {             \
    AttnLaunch b = a;                                                           \
    b.fpos = make_field_pos();                                                  \
    dim3 grid((a.n_wg > 0 ? a.n_wg : 1) * a.H * a.B);                           \
    hipLaunchKernelGGL((attn_kernel<FAM, NA, MAXB>), grid, dim3(kThreads), lds, \
                       s, b);                                                   \
    return hipGetLastError();                                                   \
  }                                                                             \
  }
