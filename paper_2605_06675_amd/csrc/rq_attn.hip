// Decode attention over the packed mixed-bit cache.
//
// Grid (workgroup slot, kv-head, batch), four waves per workgroup.  Slots
// 0 .. n_wg-1 stream the quantized 32-token blocks of their (batch, kv-head)
// unit; slot n_wg handles the 16-bit residual window.  Per block a wave:
//   QK^T on MFMA 16x16x32 f16: A = dequantized keys (16 tokens x 32
//   channels per lane quarter), B = the G query rows of this kv-head;
//   online softmax in the log2 domain (scale * log2(e) folded into q);
//   PV on MFMA 16x16x32 f16: A = probabilities (G rows x 32 tokens),
//   B = dequantized values (32 tokens x 16 channels).
// The packed format keeps codes i and i+16 of a chunk in one word, so a
// word yields an fp16 pair with one mask, and the QK result registers are
// already in the A layout PV needs.  The next block's codes and metadata
// are loaded while the current one is computed; metadata goes through LDS.
// A workgroup merges its four waves in LDS and writes one partial
// (max, sum, acc); a second kernel merges each unit's partials and writes
// the output (QuaRot: rotated back).
#include "rq_device.h"
#include "rq_internal.h"

namespace rq {

namespace {

constexpr int kWave = 64;
constexpr int kWaves = 4;
constexpr int kThreads = kWave * kWaves;
constexpr float kInvSqrtD = 0.08838834764831845f;

__device__ __forceinline__ h8 make_h8(uint32_t a, uint32_t b, uint32_t c,
                                      uint32_t d) {
  u4 v = {a, b, c, d};
  return __builtin_bit_cast(h8, v);
}

__device__ __forceinline__ f4 mfma(h8 a, h8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float xor_shfl(float v, int mask) {
  return __shfl_xor(v, mask, kWave);
}

// A block's data is four contiguous byte ranges: K codes (512*BK), V codes
// (512*BV), K metadata and V metadata (512 B each for KIVI, 64 B for
// QuaRot).  A wave moves it global -> registers -> LDS as 16-byte pieces:
// piece k of lane l covers bytes [16 l + 1024 k, +16) of the concatenation,
// so every load instruction reads 1 KB of contiguous memory.
template <int BK, int BV, bool QUAROT> struct Slot {
  static constexpr int kb = 512 * BK;
  static constexpr int vb = 512 * BV;
  static constexpr int mb = QUAROT ? 64 : 512;
  static constexpr int bytes = kb + vb + 2 * mb;
  static constexpr int pieces = (bytes + 1023) / 1024;
};

struct Ctx {
  const uint8_t* kreg;    // K codes of this unit
  const uint8_t* vreg;    // V codes of this unit
  const uint8_t* kmeta;   // K metadata of this unit
  const uint8_t* vmeta;   // V metadata of this unit
  int r, col, lane;
};

template <int BK, int BV, bool QUAROT>
__device__ __forceinline__ void load_block(const Ctx& c, int blk,
                                           u4 (&reg)[Slot<BK, BV, QUAROT>::pieces]) {
  using S = Slot<BK, BV, QUAROT>;
#pragma unroll
  for (int k = 0; k < S::pieces; ++k) {
    const int o = 16 * c.lane + 1024 * k;
    if (o < S::bytes) {
      const uint8_t* src;
      if (o < S::kb) src = c.kreg + (size_t)blk * S::kb + o;
      else if (o < S::kb + S::vb) src = c.vreg + (size_t)blk * S::vb + (o - S::kb);
      else if (o < S::kb + S::vb + S::mb) src = c.kmeta + (size_t)blk * S::mb + (o - S::kb - S::vb);
      else src = c.vmeta + (size_t)blk * S::mb + (o - S::kb - S::vb - S::mb);
      reg[k] = *reinterpret_cast<const u4*>(src);
    }
  }
}

template <int BK, int BV, bool QUAROT>
__device__ __forceinline__ void store_block(uint8_t* slot, int lane,
                                            const u4 (&reg)[Slot<BK, BV, QUAROT>::pieces]) {
  using S = Slot<BK, BV, QUAROT>;
#pragma unroll
  for (int k = 0; k < S::pieces; ++k) {
    const int o = 16 * lane + 1024 * k;
    if (o < S::bytes) *reinterpret_cast<u4*>(slot + o) = reg[k];
  }
}

// pairs i' = 0..3 (codes 4r+i' and 16+4r+i') of channel chunk `ch` (its B
// words in LDS), or'ed into the fp16 exponent pattern mg (see pair_or)
template <int BV>
__device__ __forceinline__ void vpairs(const uint32_t* ch, int r, uint32_t mg,
                                       uint32_t out[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = mg;
  int wb = 0, o = 0;
#pragma unroll
  for (int p = 0; p < Planes<BV>::n; ++p) {
    const int w = Planes<BV>::w[p];
    const uint32_t m = (((1u << w) - 1u) * 0x00010001u) << o;
    if (w == 8) {
      const uint32_t a = ch[wb + 2 * r], b = ch[wb + 2 * r + 1];
      out[0] = (shr_signed(a, -o) & m) | out[0];
      out[1] = (shr_signed(a, 8 - o) & m) | out[1];
      out[2] = (shr_signed(b, -o) & m) | out[2];
      out[3] = (shr_signed(b, 8 - o) & m) | out[3];
    } else if (w == 4) {
      const uint32_t a = ch[wb + r];
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] = (shr_signed(a, 4 * i - o) & m) | out[i];
    } else if (w == 2) {
      const uint32_t a = ch[wb + (r >> 1)] >> (8 * (r & 1));
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] = (shr_signed(a, 2 * i - o) & m) | out[i];
    } else {
      const uint32_t a = ch[wb] >> (4 * r);
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] = (shr_signed(a, i - o) & m) | out[i];
    }
    wb += w;
    o += w;
  }
}

struct WaveState {
  f4 acc[8];
  float m_run, l_run;
};

// One block, read from the LDS slot: QK^T, online softmax, PV.
template <int BK, int BV, bool QUAROT>
__device__ __forceinline__ void block_step(const Ctx& c, const uint8_t* slot,
                                           const u4* qb, WaveState& ws) {
  using S = Slot<BK, BV, QUAROT>;
  const int r = c.r;
  const uint32_t mg = opaque_magic();
  const uint32_t* kwb = reinterpret_cast<const uint32_t*>(slot);
  const uint32_t* vwb = reinterpret_cast<const uint32_t*>(slot + S::kb);
  const u4* km = reinterpret_cast<const u4*>(slot + S::kb + S::vb);
  const u4* vm = reinterpret_cast<const u4*>(slot + S::kb + S::vb + S::mb);
  uint32_t kw[2][BK];
#pragma unroll
  for (int tile = 0; tile < 2; ++tile)
#pragma unroll
    for (int i = 0; i < BK; ++i) kw[tile][i] = kwb[((16 * tile + c.col) * 4 + r) * BK + i];
  f4 S0 = {0.f, 0.f, 0.f, 0.f}, S1 = {0.f, 0.f, 0.f, 0.f};
  if (QUAROT) {
    const _Float16 o = (_Float16)(1024.0f + (float)(1 << (BK - 1)));
    const h2 off = {o, o};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const h8 qv = __builtin_bit_cast(h8, qb[kb * kWave]);
#pragma unroll
      for (int tile = 0; tile < 2; ++tile) {
        uint32_t x[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          x[kk] = as_u32(magic_to_h2(pair_or<BK>(kw[tile], 4 * kb + kk, mg), off));
        if (tile == 0) S0 = mfma(make_h8(x[0], x[1], x[2], x[3]), qv, S0);
        else S1 = mfma(make_h8(x[0], x[1], x[2], x[3]), qv, S1);
      }
    }
    // dword (4r + i) of the pair-ordered token scales = (s[4r+i], s[16+4r+i])
    const u4 sv = km[r];
    const uint32_t ss[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const h2 sc = as_h2(ss[i]);
      S0[i] *= (float)sc.x;
      S1[i] *= (float)sc.y;
    }
  } else {
    const h2 off = {(_Float16)1024.0f, (_Float16)1024.0f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const u4 s4 = km[r * 8 + kb], z4 = km[r * 8 + 4 + kb];
      const uint32_t sp[4] = {s4.x, s4.y, s4.z, s4.w};
      const uint32_t zp[4] = {z4.x, z4.y, z4.z, z4.w};
      const h8 qv = __builtin_bit_cast(h8, qb[kb * kWave]);
#pragma unroll
      for (int tile = 0; tile < 2; ++tile) {
        uint32_t x[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const h2 u = magic_to_h2(pair_or<BK>(kw[tile], 4 * kb + kk, mg), off);
          x[kk] = as_u32(__builtin_elementwise_fma(u, as_h2(sp[kk]), as_h2(zp[kk])));
        }
        if (tile == 0) S0 = mfma(make_h8(x[0], x[1], x[2], x[3]), qv, S0);
        else S1 = mfma(make_h8(x[0], x[1], x[2], x[3]), qv, S1);
      }
    }
  }
  // keep the phases apart: hoisting all LDS reads of the block to its top
  // would need more registers than four waves per SIMD allow
  __builtin_amdgcn_sched_barrier(0);
  // Online softmax in the log2 domain, column col = query row j, tokens
  // 4r+i and 16+4r+i.  The running max only moves when a block exceeds it
  // by more than 2^8 (or on the wave's first block): probabilities stay
  // <= 256, well inside fp16, and the accumulator rescale is rare.
  float mx = __builtin_fmaxf(S0[0], S1[0]);
#pragma unroll
  for (int i = 1; i < 4; ++i) mx = __builtin_fmaxf(mx, __builtin_fmaxf(S0[i], S1[i]));
  if (__builtin_amdgcn_ballot_w64(!(mx <= ws.m_run + 8.0f))) {
    mx = __builtin_fmaxf(mx, xor_shfl(mx, 16));
    mx = __builtin_fmaxf(mx, xor_shfl(mx, 32));
    const float mnew = __builtin_fmaxf(ws.m_run, mx);
    const float alpha = __builtin_amdgcn_exp2f(ws.m_run - mnew);
    ws.m_run = mnew;
    ws.l_run *= alpha;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float ar = __shfl(alpha, 4 * r + i, kWave);
#pragma unroll
      for (int nt = 0; nt < 8; ++nt) ws.acc[nt][i] *= ar;
    }
  }
  float p0[4], p1[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    p0[i] = __builtin_amdgcn_exp2f(S0[i] - ws.m_run);
    p1[i] = __builtin_amdgcn_exp2f(S1[i] - ws.m_run);
    ws.l_run += p0[i] + p1[i];
  }
  uint32_t pp[4];
  if (QUAROT) {
    const u4 sv = vm[r];
    const uint32_t ss[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const h2 sc = as_h2(ss[i]);
      const h2 pv = {(_Float16)(p0[i] * (float)sc.x), (_Float16)(p1[i] * (float)sc.y)};
      pp[i] = as_u32(pv);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const h2 pv = {(_Float16)p0[i], (_Float16)p1[i]};
      pp[i] = as_u32(pv);
    }
  }
  const h8 P = make_h8(pp[0], pp[1], pp[2], pp[3]);
  __builtin_amdgcn_sched_barrier(0);
  if (QUAROT) {
    const _Float16 o = (_Float16)(1024.0f + (float)(1 << (BV - 1)));
    const h2 off = {o, o};
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) {
      uint32_t pr[4];
      vpairs<BV>(vwb + (16 * nt + c.col) * BV, r, mg, pr);
      ws.acc[nt] = mfma(P,
                        make_h8(as_u32(magic_to_h2(pr[0], off)),
                                as_u32(magic_to_h2(pr[1], off)),
                                as_u32(magic_to_h2(pr[2], off)),
                                as_u32(magic_to_h2(pr[3], off))),
                        ws.acc[nt]);
    }
  } else {
    const h2 off = {(_Float16)1024.0f, (_Float16)1024.0f};
#pragma unroll
    for (int cg = 0; cg < 4; ++cg) {
      const u4 s4 = vm[cg * 8 + r], z4 = vm[cg * 8 + 4 + r];
      const uint32_t sp[4] = {s4.x, s4.y, s4.z, s4.w};
      const uint32_t zp[4] = {z4.x, z4.y, z4.z, z4.w};
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int nt = 2 * cg + half;
        uint32_t pr[4], x[4];
        vpairs<BV>(vwb + (16 * nt + c.col) * BV, r, mg, pr);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const h2 u = magic_to_h2(pr[i], off);
          x[i] = as_u32(__builtin_elementwise_fma(u, as_h2(sp[i]), as_h2(zp[i])));
        }
        ws.acc[nt] = mfma(P, make_h8(x[0], x[1], x[2], x[3]), ws.acc[nt]);
      }
    }
  }
}

// The wave's blocks blk_lo, blk_lo + 4, ... < blk_hi.  Two blocks are in
// flight in registers while the current one, copied into this wave's LDS
// slot, is computed.
template <int BK, int BV, bool QUAROT>
__device__ __forceinline__ void stream_blocks(const Ctx& c, int blk_lo, int blk_hi,
                                              uint8_t* slot, const u4* qb,
                                              WaveState& ws) {
  using S = Slot<BK, BV, QUAROT>;
  if (blk_lo >= blk_hi) return;
  u4 ra[S::pieces], rb[S::pieces];
  load_block<BK, BV, QUAROT>(c, blk_lo, ra);
  if (blk_lo + kWaves < blk_hi) load_block<BK, BV, QUAROT>(c, blk_lo + kWaves, rb);
  for (int blk = blk_lo; blk < blk_hi; blk += 2 * kWaves) {
    store_block<BK, BV, QUAROT>(slot, c.lane, ra);
    if (blk + 2 * kWaves < blk_hi) load_block<BK, BV, QUAROT>(c, blk + 2 * kWaves, ra);
    block_step<BK, BV, QUAROT>(c, slot, qb, ws);
    const int b1 = blk + kWaves;
    if (b1 >= blk_hi) break;
    store_block<BK, BV, QUAROT>(slot, c.lane, rb);
    if (b1 + 2 * kWaves < blk_hi) load_block<BK, BV, QUAROT>(c, b1 + 2 * kWaves, rb);
    block_step<BK, BV, QUAROT>(c, slot, qb, ws);
  }
}

template <bool QUAROT, int MAXB>
__device__ __forceinline__ void dispatch(int bk, int bv, const Ctx& c, int lo, int hi,
                                         uint8_t* slot, const u4* qb, WaveState& ws) {
#define RQ_CASE(K, V)                                                   \
  case (K - 1) * 8 + (V - 1):                                           \
    if (K <= MAXB && V <= MAXB)                                         \
      stream_blocks<(K <= MAXB ? K : 1), (V <= MAXB ? V : 1), QUAROT>(   \
          c, lo, hi, slot, qb, ws);                                     \
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

// Scaled query rows of this kv-head into qs (rows >= G zero), rotated for
// QuaRot.  Whole workgroup.
__device__ __forceinline__ void load_queries(const AttnLaunch& a, int b, int h, bool rotate,
                             float (*qs)[kD]) {
  const int tid = threadIdx.x;
  for (int e = tid; e < 16 * kD; e += kThreads) {
    const int j = e / kD, cc = e % kD;
    float v = 0.0f;
    if (j < a.G)
      v = widen(a.q[((size_t)b * a.H * a.G + h * a.G + j) * kD + cc], a.is_bf16);
    qs[j][cc] = v;
  }
  __syncthreads();
  float f = a.qscale;
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
    f *= kInvSqrtD;
  }
  for (int e = tid; e < a.G * kD; e += kThreads) qs[e / kD][e % kD] *= f;
  __syncthreads();
}

// Partial of (unit, slot): float [G][2 + 128] = (max, sum, acc[128]).
__device__ __forceinline__ float* part_ptr(const AttnLaunch& a, size_t unit,
                                           int slot) {
  return a.part + (unit * (a.n_wg + 1) + slot) * (size_t)a.G * (2 + kD);
}

// 16-bit residual window of one unit, original domain; wave w takes query
// rows w, w+4, ...; lane = token for scores, lane = channel pair for PV.
__device__ __forceinline__ void residual_slot(const AttnLaunch& a, int b, int h,
                              const float (*qs)[kD], float* dst) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
  const int cap = a.R + kChunk;
  const uint16_t* kb = a.resid + (((size_t)b * a.H + h) * 2 + 0) * cap * kD;
  const uint16_t* vb = a.resid + (((size_t)b * a.H + h) * 2 + 1) * cap * kD;
  for (int j = wave; j < a.G; j += kWaves) {
    float m_run = -INFINITY, l_run = 0.0f, ac0 = 0.0f, ac1 = 0.0f;
    for (int t0 = a.nq; t0 < a.n_tokens; t0 += kWave) {
      const int t = t0 + lane;
      const bool ok = t < a.n_tokens;
      float s = -INFINITY;
      if (ok) {
        const uint16_t* kr = kb + (size_t)(t % cap) * kD;
        s = 0.0f;
        for (int cc = 0; cc < kD; cc += 2) {
          const uint32_t w = *reinterpret_cast<const uint32_t*>(kr + cc);
          s = __builtin_fmaf(qs[j][cc], widen(w & 0xffffu, a.is_bf16), s);
          s = __builtin_fmaf(qs[j][cc + 1], widen(w >> 16, a.is_bf16), s);
        }
      }
      float mx = s;
      for (int d = 32; d >= 1; d >>= 1) mx = __builtin_fmaxf(mx, xor_shfl(mx, d));
      const float mn = __builtin_fmaxf(m_run, mx);
      const float al = __builtin_amdgcn_exp2f(m_run - mn);
      const float p = ok ? __builtin_amdgcn_exp2f(s - mn) : 0.0f;
      float sum = p;
      for (int d = 32; d >= 1; d >>= 1) sum += xor_shfl(sum, d);
      l_run = l_run * al + sum;
      m_run = mn;
      ac0 *= al;
      ac1 *= al;
      const int n = (a.n_tokens - t0) < kWave ? (a.n_tokens - t0) : kWave;
      for (int i = 0; i < n; ++i) {
        const uint32_t w = *reinterpret_cast<const uint32_t*>(
            vb + (size_t)((t0 + i) % cap) * kD + 2 * lane);
        const float pi = __shfl(p, i, kWave);
        ac0 = __builtin_fmaf(pi, widen(w & 0xffffu, a.is_bf16), ac0);
        ac1 = __builtin_fmaf(pi, widen(w >> 16, a.is_bf16), ac1);
      }
    }
    float* d = dst + (size_t)j * (2 + kD);
    if (lane == 0) {
      d[0] = m_run;
      d[1] = l_run;
    }
    d[2 + 2 * lane] = ac0;
    d[2 + 2 * lane + 1] = ac1;
  }
}

// MAXB: largest bit-width the kernel handles (4: the common {1..4} range,
// compiled for three resident waves per SIMD, each with two blocks in
// flight; 8: every width).
template <int MAXB>
__global__ void __launch_bounds__(kThreads, MAXB <= 4 ? 3 : 2)
attn_kernel(AttnLaunch a) {
  __shared__ float qs[16][kD];
  __shared__ u4 qbuf[4][kWave];      // QK B operand per (K-block, lane)
  // per-wave block slots while streaming, then the wave merge area
  // [kWaves][G][2 + 128] floats
  extern __shared__ u4 dyn[];
  uint8_t* slots = reinterpret_cast<uint8_t*>(dyn);
  float* merge = reinterpret_cast<float*>(dyn);
  const int slot = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid & (kWave - 1);
  const size_t unit = (size_t)b * a.H + h;
  const bool quarot = a.family == RQ_QUAROT;
  const int G = a.G;

  if (slot == a.n_wg) {
    load_queries(a, b, h, false, qs);
    residual_slot(a, b, h, qs, part_ptr(a, unit, slot));
  } else {
    load_queries(a, b, h, quarot, qs);
    const int r = lane >> 4, col = lane & 15;
    // B operand of QK: column j = col, k-slots of quarter r, K-block kb:
    // channels 32r + 4kb + k' and 32r + 16 + 4kb + k', k' = 0..3
    if (wave == 0) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        uint32_t x[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int c0 = 32 * r + 4 * kb + kk;
          const h2 v = {(_Float16)qs[col][c0], (_Float16)qs[col][c0 + 16]};
          x[kk] = as_u32(v);
        }
        qbuf[kb][lane] = (u4){x[0], x[1], x[2], x[3]};
      }
    }
    __syncthreads();
    const u4* qb = &qbuf[0][lane];
    const int bk = a.tab.bits[h][0], bv = a.tab.bits[h][1];
    const int nblk_cap = a.cap / kChunk;
    const int per_blk = quarot ? kMetaBlockTok : kMetaBlockKivi;
    Ctx c;
    c.kreg = a.codes + a.tab.code_off[h][0] + (size_t)b * a.cap * 16 * bk;
    c.vreg = a.codes + a.tab.code_off[h][1] + (size_t)b * a.cap * 16 * bv;
    c.kmeta = a.meta + (((size_t)h * 2 + 0) * a.B + b) * nblk_cap * per_blk;
    c.vmeta = a.meta + (((size_t)h * 2 + 1) * a.B + b) * nblk_cap * per_blk;
    c.r = r;
    c.col = col;
    c.lane = lane;
    WaveState ws;
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) ws.acc[nt] = (f4){0.f, 0.f, 0.f, 0.f};
    ws.m_run = -INFINITY;
    ws.l_run = 0.0f;
    const int nblk = a.nq / kChunk;
    const int lo = slot * a.blk_per_wg;
    int hi = lo + a.blk_per_wg;
    if (hi > nblk) hi = nblk;
    uint8_t* my_slot = slots + (size_t)wave * a.slot_bytes;
    if (quarot)
      dispatch<true, MAXB>(bk, bv, c, lo + wave, hi, my_slot, qb, ws);
    else
      dispatch<false, MAXB>(bk, bv, c, lo + wave, hi, my_slot, qb, ws);
    ws.l_run += xor_shfl(ws.l_run, 16);
    ws.l_run += xor_shfl(ws.l_run, 32);
    // merge the four waves in LDS (the merge area reuses the block slots)
    __syncthreads();
    float* mw = merge + (size_t)wave * G * (2 + kD);
    if (r == 0 && col < G) {
      mw[col * (2 + kD)] = ws.m_run;
      mw[col * (2 + kD) + 1] = ws.l_run;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = 4 * r + i;
      if (j < G) {
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) mw[j * (2 + kD) + 2 + 16 * nt + col] = ws.acc[nt][i];
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
        const float f = (M == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(src[0] - M);
        acc = __builtin_fmaf(f, src[2 + cc], acc);
        l = __builtin_fmaf(f, src[1], l);
      }
      dst[j * (2 + kD) + 2 + cc] = acc;
      if (cc == 0) {
        dst[j * (2 + kD)] = M;
        dst[j * (2 + kD) + 1] = l;
      }
    }
  }

}

// Merge the partials of one (batch, kv-head) unit: one workgroup per unit.
// Slots 0 .. n_wg-1 hold the quantized blocks (QuaRot: rotated domain),
// slot n_wg the 16-bit window (original domain).  All loads of a stage are
// independent, so they are in flight together.
__global__ void __launch_bounds__(kThreads)
combine_kernel(AttnLaunch a) {
  extern __shared__ float lds[];   // wgt[ns][G], lsum[ns][G], rot[G][128]
  const int unit = blockIdx.x, tid = threadIdx.x;
  const int G = a.G;
  const bool quarot = a.family == RQ_QUAROT;
  const int ns = a.n_wg + 1;
  float* wgt = lds;
  float* lsum = lds + ns * G;
  float* rot = lds + 2 * ns * G;
  __shared__ float inv_den[16];
  // per (slot, j): max and sum, then weights relative to the row max
  for (int e = tid; e < ns * G; e += kThreads) {
    const float* src = part_ptr(a, unit, e / G) + (e % G) * (2 + kD);
    wgt[e] = src[1] > 0.0f ? src[0] : -INFINITY;
    lsum[e] = src[1];
  }
  __syncthreads();
  if (tid < G) {
    float M = -INFINITY;
    for (int sl = 0; sl < ns; ++sl) M = __builtin_fmaxf(M, wgt[sl * G + tid]);
    float den = 0.0f;
    for (int sl = 0; sl < ns; ++sl) {
      const float m = wgt[sl * G + tid];
      const float f = m == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(m - M);
      wgt[sl * G + tid] = f;
      den = __builtin_fmaf(f, lsum[sl * G + tid], den);
    }
    inv_den[tid] = 1.0f / den;
  }
  __syncthreads();
  float tailv[(16 * kD) / kThreads];
  int n_e = 0;
  for (int e = tid; e < G * kD; e += kThreads, ++n_e) {
    const int j = e / kD, cc = e % kD;
    float num = 0.0f;
    const float* src = part_ptr(a, unit, 0) + j * (2 + kD) + 2 + cc;
    const size_t stride = (size_t)G * (2 + kD);
#pragma unroll 8
    for (int sl = 0; sl < ns - 1; ++sl) num = __builtin_fmaf(wgt[sl * G + j], src[sl * stride], num);
    tailv[n_e] = wgt[(ns - 1) * G + j] * src[(ns - 1) * stride];
    rot[e] = num;
  }
  __syncthreads();
  if (quarot) {
    for (int hh = 1; hh < kD; hh *= 2) {
      for (int e = tid; e < G * (kD / 2); e += kThreads) {
        const int j = e / (kD / 2), i = e % (kD / 2);
        const int base = (i / hh) * 2 * hh + (i % hh);
        const float x = rot[j * kD + base], y = rot[j * kD + base + hh];
        rot[j * kD + base] = x + y;
        rot[j * kD + base + hh] = x - y;
      }
      __syncthreads();
    }
  }
  const float f = quarot ? kInvSqrtD : 1.0f;
  float* out = a.out + (size_t)unit * G * kD;   // (b, h) -> query rows h*G..
  n_e = 0;
  for (int e = tid; e < G * kD; e += kThreads, ++n_e)
    out[e] = (rot[e] * f + tailv[n_e]) * inv_den[e / kD];
}

}  // namespace

size_t attention_lds_bytes(int G, int slot_bytes) {
  const size_t merge = (size_t)kWaves * G * (2 + kD) * sizeof(float);
  const size_t slots = (size_t)kWaves * slot_bytes;
  return merge > slots ? merge : slots;
}

hipError_t launch_attention(const AttnLaunch& a, hipStream_t s) {
  dim3 grid(a.n_wg + 1, a.H, a.B);
  int maxb = 1;
  for (int h = 0; h < a.H; ++h)
    for (int k = 0; k < 2; ++k) maxb = a.tab.bits[h][k] > maxb ? a.tab.bits[h][k] : maxb;
  if (maxb <= 4)
    hipLaunchKernelGGL(attn_kernel<4>, grid, dim3(kThreads),
                       attention_lds_bytes(a.G, a.slot_bytes), s, a);
  else
    hipLaunchKernelGGL(attn_kernel<8>, grid, dim3(kThreads),
                       attention_lds_bytes(a.G, a.slot_bytes), s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds = ((size_t)2 * (a.n_wg + 1) * a.G + (size_t)a.G * kD) * sizeof(float);
  hipLaunchKernelGGL(combine_kernel, dim3(a.B * a.H), dim3(kThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace rq
