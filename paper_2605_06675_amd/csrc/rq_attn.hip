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

// Words of a V chunk that lane quarter r needs, per plane: 2 for the 8-bit
// plane, 1 otherwise.
template <int B> struct VWords {
  static constexpr int n = (B == 8) ? 2 : Planes<B>::n;
};

template <int BK> struct KStage {
  uint32_t kw[2][BK];
  u4 meta;
};

template <int BV> struct VStage {
  uint32_t vw[8][VWords<BV>::n];
};

struct Ctx {
  const uint32_t* kreg;   // K codes of this unit
  const uint32_t* vreg;   // V codes of this unit
  const uint8_t* kmeta;   // K metadata of this unit
  const uint8_t* vmeta;   // V metadata of this unit
  int per_blk;            // metadata bytes per block and kind
  int r, col, lane;
};

// K words of the block (tiles 0/1: token 16*tile + col, chunk r) and this
// lane's 16 bytes of the block metadata (lanes 0..31: K, 32..63: V).
template <int BK>
__device__ __forceinline__ void fetch_k(const Ctx& c, int blk, KStage<BK>& s) {
#pragma unroll
  for (int tile = 0; tile < 2; ++tile) {
    const uint32_t* p = c.kreg + ((size_t)(blk * kChunk + 16 * tile + c.col) * 4 + c.r) * BK;
#pragma unroll
    for (int i = 0; i < BK; ++i) s.kw[tile][i] = p[i];
  }
  const int half = c.lane >> 5, i = c.lane & 31;
  if (i * 16 < c.per_blk) {
    const uint8_t* m = (half ? c.vmeta : c.kmeta) + (size_t)blk * c.per_blk + i * 16;
    s.meta = *reinterpret_cast<const u4*>(m);
  }
}

// V words lane quarter r needs from the chunks of channels 16*nt + col.
template <int BV>
__device__ __forceinline__ void fetch_v(const Ctx& c, int blk, VStage<BV>& s) {
  const uint32_t* base = c.vreg + ((size_t)blk * kD + c.col) * BV;
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) {
    const uint32_t* ch = base + 16 * nt * BV;
    int wb = 0, k = 0;
#pragma unroll
    for (int p = 0; p < Planes<BV>::n; ++p) {
      const int w = Planes<BV>::w[p];
      if (w == 8) {
        s.vw[nt][k++] = ch[wb + 2 * c.r];
        s.vw[nt][k++] = ch[wb + 2 * c.r + 1];
      } else if (w == 4) {
        s.vw[nt][k++] = ch[wb + c.r];
      } else if (w == 2) {
        s.vw[nt][k++] = ch[wb + (c.r >> 1)];
      } else {
        s.vw[nt][k++] = ch[wb];
      }
      wb += w;
    }
  }
}

// pairs i' = 0..3 (codes 4r+i' and 16+4r+i') of the lane's V chunk words,
// or'ed into the fp16 exponent pattern mg (see pair_or)
template <int BV>
__device__ __forceinline__ void vpairs(const uint32_t* vw, int r, uint32_t mg,
                                       uint32_t out[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = mg;
  int k = 0, o = 0;
#pragma unroll
  for (int p = 0; p < Planes<BV>::n; ++p) {
    const int w = Planes<BV>::w[p];
    const uint32_t m = (((1u << w) - 1u) * 0x00010001u) << o;
    if (w == 8) {
      const uint32_t a = vw[k], b = vw[k + 1];
      out[0] = (shr_signed(a, -o) & m) | out[0];
      out[1] = (shr_signed(a, 8 - o) & m) | out[1];
      out[2] = (shr_signed(b, -o) & m) | out[2];
      out[3] = (shr_signed(b, 8 - o) & m) | out[3];
      k += 2;
    } else if (w == 4) {
      const uint32_t a = vw[k++];
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] = (shr_signed(a, 4 * i - o) & m) | out[i];
    } else if (w == 2) {
      const uint32_t a = vw[k++] >> (8 * (r & 1));
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] = (shr_signed(a, 2 * i - o) & m) | out[i];
    } else {
      const uint32_t a = vw[k++] >> (4 * r);
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] = (shr_signed(a, i - o) & m) | out[i];
    }
    o += w;
  }
}

struct WaveState {
  f4 acc[8];
  float m_run, l_run;
};

// One block: QK^T, online softmax, PV.  mb = this wave's metadata in LDS
// (u4 index 0.. = K metadata, 32.. = V metadata).
template <int BK, int BV, bool QUAROT>
__device__ __forceinline__ void block_step(const Ctx& c, KStage<BK>& s,
                                           VStage<BV>& sv_, const u4* mb,
                                           const u4* qb, WaveState& ws,
                                           bool more, int nb) {
  const int r = c.r;
  const uint32_t mg = opaque_magic();
  f4 S0 = {0.f, 0.f, 0.f, 0.f}, S1 = {0.f, 0.f, 0.f, 0.f};
  if (QUAROT) {
    const _Float16 o = (_Float16)(1024.0f + (float)(1 << (BK - 1)));
    const h2 off = {o, o};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
      for (int tile = 0; tile < 2; ++tile) {
        uint32_t x[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          x[kk] = as_u32(magic_to_h2(pair_or<BK>(s.kw[tile], 4 * kb + kk, mg), off));
        const h8 qv = __builtin_bit_cast(h8, qb[kb * kWave]);
        if (tile == 0) S0 = mfma(make_h8(x[0], x[1], x[2], x[3]), qv, S0);
        else S1 = mfma(make_h8(x[0], x[1], x[2], x[3]), qv, S1);
      }
    }
    const u4 sv = mb[r];
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
      const u4 s4 = mb[r * 8 + kb], z4 = mb[r * 8 + 4 + kb];
      const uint32_t sp[4] = {s4.x, s4.y, s4.z, s4.w};
      const uint32_t zp[4] = {z4.x, z4.y, z4.z, z4.w};
#pragma unroll
      for (int tile = 0; tile < 2; ++tile) {
        uint32_t x[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const h2 u = magic_to_h2(pair_or<BK>(s.kw[tile], 4 * kb + kk, mg), off);
          x[kk] = as_u32(__builtin_elementwise_fma(u, as_h2(sp[kk]), as_h2(zp[kk])));
        }
        const h8 qv = __builtin_bit_cast(h8, qb[kb * kWave]);
        if (tile == 0) S0 = mfma(make_h8(x[0], x[1], x[2], x[3]), qv, S0);
        else S1 = mfma(make_h8(x[0], x[1], x[2], x[3]), qv, S1);
      }
    }
  }
  if (more) fetch_k<BK>(c, nb, s);
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
    const u4 sv = mb[32 + r];
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
  if (QUAROT) {
    const _Float16 o = (_Float16)(1024.0f + (float)(1 << (BV - 1)));
    const h2 off = {o, o};
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) {
      uint32_t pr[4];
      vpairs<BV>(sv_.vw[nt], r, mg, pr);
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
      const u4 s4 = mb[32 + cg * 8 + r], z4 = mb[32 + cg * 8 + 4 + r];
      const uint32_t sp[4] = {s4.x, s4.y, s4.z, s4.w};
      const uint32_t zp[4] = {z4.x, z4.y, z4.z, z4.w};
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int nt = 2 * cg + half;
        uint32_t pr[4], x[4];
        vpairs<BV>(sv_.vw[nt], r, mg, pr);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const h2 u = magic_to_h2(pr[i], off);
          x[i] = as_u32(__builtin_elementwise_fma(u, as_h2(sp[i]), as_h2(zp[i])));
        }
        ws.acc[nt] = mfma(P, make_h8(x[0], x[1], x[2], x[3]), ws.acc[nt]);
      }
    }
  }
  if (more) fetch_v<BV>(c, nb, sv_);
}

template <int BK, int BV, bool QUAROT>
__device__ __forceinline__ void stream_blocks(const Ctx& c, int blk_lo, int blk_hi,
                                              u4* mb, const u4* qb, WaveState& ws) {
  if (blk_lo >= blk_hi) return;
  // Single-buffered pipeline: the next block's K words (+ metadata) are
  // requested as soon as QK^T has consumed this block's, and its V words
  // as soon as PV has consumed this block's.
  KStage<BK> ks;
  VStage<BV> vs;
  fetch_k<BK>(c, blk_lo, ks);
  fetch_v<BV>(c, blk_lo, vs);
  for (int blk = blk_lo; blk < blk_hi; blk += kWaves) {
    mb[c.lane] = ks.meta;
    const int nb = blk + kWaves;
    block_step<BK, BV, QUAROT>(c, ks, vs, mb, qb, ws, nb < blk_hi, nb);
  }
}

template <bool QUAROT, int MAXB>
__device__ __forceinline__ void dispatch(int bk, int bv, const Ctx& c, int lo, int hi, u4* mb,
                         const u4* qb, WaveState& ws) {
#define RQ_CASE(K, V)                                                   \
  case (K - 1) * 8 + (V - 1):                                           \
    if (K <= MAXB && V <= MAXB)                                         \
      stream_blocks<(K <= MAXB ? K : 1), (V <= MAXB ? V : 1), QUAROT>(   \
          c, lo, hi, mb, qb, ws);                                       \
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
// compiled for four resident waves per SIMD; 8: every width).
template <int MAXB>
__global__ void __launch_bounds__(kThreads, MAXB <= 4 ? 4 : 2)
attn_kernel(AttnLaunch a) {
  __shared__ float qs[16][kD];
  __shared__ u4 mbuf[kWaves][kWave];
  __shared__ u4 qbuf[4][kWave];      // QK B operand per (K-block, lane)
  extern __shared__ float merge[];   // [kWaves][G][2 + 128]
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
    Ctx c;
    c.per_blk = quarot ? kMetaBlockTok : kMetaBlockKivi;
    c.kreg = reinterpret_cast<const uint32_t*>(a.codes + a.tab.code_off[h][0]) +
             (size_t)b * a.cap * 4 * bk;
    c.vreg = reinterpret_cast<const uint32_t*>(a.codes + a.tab.code_off[h][1]) +
             (size_t)b * nblk_cap * kD * bv;
    c.kmeta = a.meta + (((size_t)h * 2 + 0) * a.B + b) * nblk_cap * c.per_blk;
    c.vmeta = a.meta + (((size_t)h * 2 + 1) * a.B + b) * nblk_cap * c.per_blk;
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
    if (quarot)
      dispatch<true, MAXB>(bk, bv, c, lo + wave, hi, mbuf[wave], qb, ws);
    else
      dispatch<false, MAXB>(bk, bv, c, lo + wave, hi, mbuf[wave], qb, ws);
    ws.l_run += xor_shfl(ws.l_run, 16);
    ws.l_run += xor_shfl(ws.l_run, 32);
    // merge the four waves in LDS
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

size_t attention_lds_bytes(int G) {
  return (size_t)kWaves * G * (2 + kD) * sizeof(float);
}

hipError_t launch_attention(const AttnLaunch& a, hipStream_t s) {
  dim3 grid(a.n_wg + 1, a.H, a.B);
  int maxb = 1;
  for (int h = 0; h < a.H; ++h)
    for (int k = 0; k < 2; ++k) maxb = a.tab.bits[h][k] > maxb ? a.tab.bits[h][k] : maxb;
  if (maxb <= 4)
    hipLaunchKernelGGL(attn_kernel<4>, grid, dim3(kThreads),
                       attention_lds_bytes(a.G), s, a);
  else
    hipLaunchKernelGGL(attn_kernel<8>, grid, dim3(kThreads),
                       attention_lds_bytes(a.G), s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds = ((size_t)2 * (a.n_wg + 1) * a.G + (size_t)a.G * kD) * sizeof(float);
  hipLaunchKernelGGL(combine_kernel, dim3(a.B * a.H), dim3(kThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace rq
