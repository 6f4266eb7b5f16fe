// Decode attention over the packed mixed-bit cache.
//
// Grid (split group, kv-head, batch), four waves per workgroup sharing the
// query rows in LDS; each wave is one split, a run of 32-token blocks of its
// (batch, kv-head) unit:
//   QK^T on MFMA 16x16x32 f16: A = dequantized keys (16 tokens x 32
//   channels per lane-quarter), B = the G query rows of this kv-head;
//   online softmax in the log2 domain (scale * log2(e) folded into q);
//   PV on MFMA 16x16x32 f16: A = probabilities (G rows x 32 tokens),
//   B = dequantized values (32 tokens x 16 channels).
// The packed format keeps codes i and i+16 of a chunk in one word, so a
// word yields an fp16 pair with one mask, and the QK result registers are
// already in the A layout PV needs (no shuffles between the two products).
// The extra split index n_split handles the 16-bit residual window on VALU.
// Each split writes (max, sum, acc) partials; a second kernel combines them
// (and, for QuaRot, rotates the output back).
#include "rq_device.h"
#include "rq_internal.h"

namespace rq {

namespace {

constexpr int kWave = 64;
constexpr float kInvSqrtD = 0.08838834764831845f;

__device__ __forceinline__ h8 make_h8(uint32_t a, uint32_t b, uint32_t c,
                                      uint32_t d) {
  u4 v = {a, b, c, d};
  return __builtin_bit_cast(h8, v);
}

__device__ __forceinline__ f4 mfma(h8 a, h8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

template <int B>
__device__ __forceinline__ void load_words(const uint32_t* p, uint32_t w[B]) {
#pragma unroll
  for (int i = 0; i < B; ++i) w[i] = p[i];
}

// Pairs i' = 0..3 (codes 4r+i' and 16+4r+i') of a chunk, reading only the
// words lane-quarter r needs.
template <int B>
__device__ __forceinline__ void value_pairs(const uint32_t* chunk, int r,
                                            uint32_t out[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = 0;
  int wb = 0, o = 0;
#pragma unroll
  for (int p = 0; p < Planes<B>::n; ++p) {
    const int w = Planes<B>::w[p];
    const uint32_t m = ((1u << w) - 1u) * 0x00010001u;
    if (w == 8) {
      const uint32_t a = chunk[wb + 2 * r], b = chunk[wb + 2 * r + 1];
      out[0] |= (a & m) << o;
      out[1] |= ((a >> 8) & m) << o;
      out[2] |= (b & m) << o;
      out[3] |= ((b >> 8) & m) << o;
    } else if (w == 4) {
      const uint32_t a = chunk[wb + r];
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] |= ((a >> (4 * i)) & m) << o;
    } else if (w == 2) {
      const uint32_t a = chunk[wb + (r >> 1)] >> (8 * (r & 1));
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] |= ((a >> (2 * i)) & m) << o;
    } else {
      const uint32_t a = chunk[wb] >> (4 * r);
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] |= ((a >> i) & m) << o;
    }
    wb += w;
    o += w;
  }
}

struct KCtx {
  const uint32_t* region;   // K code region of this (head), batch applied
  const uint8_t* meta;      // K metadata of this unit
  int r, m;                 // lane quarter, lane row
};

// QK^T of one 32-token block, KIVI keys: K_hat = u * s + z per channel.
template <int B>
__device__ __forceinline__ void qk_kivi(const KCtx& k, int blk, const h8 qb[4],
                                        f4& S0, f4& S1) {
  const u4* mp = reinterpret_cast<const u4*>(k.meta + (size_t)blk * kMetaBlockKivi +
                                             k.r * 128);
  uint32_t sp[16], zp[16];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const u4 a = mp[i], c = mp[4 + i];
    sp[4 * i] = a.x; sp[4 * i + 1] = a.y; sp[4 * i + 2] = a.z; sp[4 * i + 3] = a.w;
    zp[4 * i] = c.x; zp[4 * i + 1] = c.y; zp[4 * i + 2] = c.z; zp[4 * i + 3] = c.w;
  }
  const h2 off = {(_Float16)1024.0f, (_Float16)1024.0f};
#pragma unroll
  for (int tile = 0; tile < 2; ++tile) {
    const int t = blk * kChunk + 16 * tile + k.m;
    uint32_t w[B];
    load_words<B>(k.region + ((size_t)t * 4 + k.r) * B, w);
    f4 S = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      uint32_t x[4];
#define RQ_KP(KK)                                                        \
      {                                                                  \
        const h2 u = codes_to_h2(pair_bits<B>(w, 4 * kb + KK), off);     \
        x[KK] = as_u32(__builtin_elementwise_fma(                        \
            u, as_h2(sp[4 * kb + KK]), as_h2(zp[4 * kb + KK])));         \
      }
      RQ_KP(0) RQ_KP(1) RQ_KP(2) RQ_KP(3)
#undef RQ_KP
      S = mfma(make_h8(x[0], x[1], x[2], x[3]), qb[kb], S);
    }
    if (tile == 0) S0 = S; else S1 = S;
  }
}

// QK^T of one block, QuaRot keys: scores of token t scaled by s_t after the
// product of q_rot with the integer levels (u - 2^(b-1)).
template <int B>
__device__ __forceinline__ void qk_quarot(const KCtx& k, int blk, const h8 qb[4],
                                          f4& S0, f4& S1) {
  const _Float16 o = (_Float16)(1024.0f + (float)(1 << (B - 1)));
  const h2 off = {o, o};
#pragma unroll
  for (int tile = 0; tile < 2; ++tile) {
    const int t = blk * kChunk + 16 * tile + k.m;
    uint32_t w[B];
    load_words<B>(k.region + ((size_t)t * 4 + k.r) * B, w);
    f4 S = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const uint32_t x0 = as_u32(codes_to_h2(pair_bits<B>(w, 4 * kb + 0), off));
      const uint32_t x1 = as_u32(codes_to_h2(pair_bits<B>(w, 4 * kb + 1), off));
      const uint32_t x2 = as_u32(codes_to_h2(pair_bits<B>(w, 4 * kb + 2), off));
      const uint32_t x3 = as_u32(codes_to_h2(pair_bits<B>(w, 4 * kb + 3), off));
      S = mfma(make_h8(x0, x1, x2, x3), qb[kb], S);
    }
    if (tile == 0) S0 = S; else S1 = S;
  }
  // per-token scales: dword (4r + i) of the block's pair-ordered scales
  // holds (s[4r + i], s[16 + 4r + i])
  const u4 sv = *reinterpret_cast<const u4*>(k.meta + (size_t)blk * kMetaBlockTok +
                                             k.r * 16);
  const uint32_t ss[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const h2 s = as_h2(ss[i]);
    S0[i] *= (float)s.x;
    S1[i] *= (float)s.y;
  }
}

struct VCtx {
  const uint32_t* region;   // V code region of this head, batch applied
  const uint8_t* meta;      // V metadata of this unit
  int r, n;
};

template <int B>
__device__ __forceinline__ void pv_kivi(const VCtx& v, int blk, const h8& P,
                                        f4 acc[8]) {
  const h2 off = {(_Float16)1024.0f, (_Float16)1024.0f};
  const uint32_t* cb = v.region + (size_t)blk * kD * B;
  const uint8_t* mb = v.meta + (size_t)blk * kMetaBlockKivi;
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) {
    const int c = 16 * nt + v.n, cg = nt >> 1;
    const u4 s4 = *reinterpret_cast<const u4*>(mb + cg * 128 + v.r * 16);
    const u4 z4 = *reinterpret_cast<const u4*>(mb + cg * 128 + 64 + v.r * 16);
    const uint32_t sp[4] = {s4.x, s4.y, s4.z, s4.w};
    const uint32_t zp[4] = {z4.x, z4.y, z4.z, z4.w};
    uint32_t pr[4];
    value_pairs<B>(cb + (size_t)c * B, v.r, pr);
    uint32_t x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const h2 u = codes_to_h2(pr[i], off);
      x[i] = as_u32(__builtin_elementwise_fma(u, as_h2(sp[i]), as_h2(zp[i])));
    }
    acc[nt] = mfma(P, make_h8(x[0], x[1], x[2], x[3]), acc[nt]);
  }
}

template <int B>
__device__ __forceinline__ void pv_quarot(const VCtx& v, int blk, const h8& P,
                                          f4 acc[8]) {
  const _Float16 o = (_Float16)(1024.0f + (float)(1 << (B - 1)));
  const h2 off = {o, o};
  const uint32_t* cb = v.region + (size_t)blk * kD * B;
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) {
    const int c = 16 * nt + v.n;
    uint32_t pr[4];
    value_pairs<B>(cb + (size_t)c * B, v.r, pr);
    acc[nt] = mfma(P,
                   make_h8(as_u32(codes_to_h2(pr[0], off)),
                           as_u32(codes_to_h2(pr[1], off)),
                           as_u32(codes_to_h2(pr[2], off)),
                           as_u32(codes_to_h2(pr[3], off))),
                   acc[nt]);
  }
}

#define RQ_DISPATCH8(bits, F, ...)          \
  switch (bits) {                           \
    case 1: F<1>(__VA_ARGS__); break;       \
    case 2: F<2>(__VA_ARGS__); break;       \
    case 3: F<3>(__VA_ARGS__); break;       \
    case 4: F<4>(__VA_ARGS__); break;       \
    case 5: F<5>(__VA_ARGS__); break;       \
    case 6: F<6>(__VA_ARGS__); break;       \
    case 7: F<7>(__VA_ARGS__); break;       \
    default: F<8>(__VA_ARGS__); break;      \
  }

__device__ __forceinline__ float xor_shfl(float v, int mask) {
  return __shfl_xor(v, mask, kWave);
}

// Fills qs[j][c] (fp32, LDS) with the scaled (and, for QuaRot, rotated)
// query rows of this kv-head; rows >= G are zero.  All threads of the
// workgroup take part.
__device__ void load_queries(const AttnLaunch& a, int b, int h, bool rotate,
                             float (*qs)[kD]) {
  const int tid = threadIdx.x, nthr = blockDim.x;
  for (int e = tid; e < 16 * kD; e += nthr) {
    const int j = e / kD, c = e % kD;
    float v = 0.0f;
    if (j < a.G)
      v = widen(a.q[((size_t)b * a.H * a.G + h * a.G + j) * kD + c], a.is_bf16);
    qs[j][c] = v;
  }
  __syncthreads();
  float f = a.qscale;
  if (rotate) {
    // q_rot = (1/sqrt(128)) H q (any butterfly order: attention tolerance)
    for (int hh = 1; hh < kD; hh *= 2) {
      for (int e = tid; e < a.G * (kD / 2); e += nthr) {
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
  for (int e = tid; e < a.G * kD; e += nthr) qs[e / kD][e % kD] *= f;
  __syncthreads();
}

// 16-bit residual window on VALU, one wave: lane = token for the scores,
// lane = channel pair for PV; probabilities move between lanes by shuffles.
// qs holds the unrotated scaled queries.
__device__ void residual_split(const AttnLaunch& a, int b, int h,
                               const float (*qs)[kD], float* ml, float* accw) {
  const int lane = threadIdx.x & (kWave - 1);
  const int cap = a.R + kChunk;
  float m_run[16], l_run[16], ac[16][2];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    m_run[j] = -INFINITY;
    l_run[j] = 0.0f;
    ac[j][0] = ac[j][1] = 0.0f;
  }
  const uint16_t* kbase = a.resid + (((size_t)b * a.H + h) * 2 + 0) * cap * kD;
  const uint16_t* vbase = a.resid + (((size_t)b * a.H + h) * 2 + 1) * cap * kD;
  for (int t0 = a.nq; t0 < a.n_tokens; t0 += kWave) {
    const int t = t0 + lane;
    const bool ok = t < a.n_tokens;
    float s[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) s[j] = 0.0f;
    if (ok) {
      const uint16_t* kr = kbase + (size_t)(t % cap) * kD;
      for (int c = 0; c < kD; c += 2) {
        const uint32_t w = *reinterpret_cast<const uint32_t*>(kr + c);
        const float k0 = widen(w & 0xffffu, a.is_bf16);
        const float k1 = widen(w >> 16, a.is_bf16);
#pragma unroll
        for (int j = 0; j < 16; ++j)
          s[j] = __builtin_fmaf(qs[j][c + 1], k1, __builtin_fmaf(qs[j][c], k0, s[j]));
      }
    }
    float p[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      p[j] = 0.0f;
      if (j < a.G) {
        float mx = ok ? s[j] : -INFINITY;
        for (int d = 32; d >= 1; d >>= 1) mx = __builtin_fmaxf(mx, xor_shfl(mx, d));
        const float mn = __builtin_fmaxf(m_run[j], mx);
        const float al = __builtin_amdgcn_exp2f(m_run[j] - mn);
        p[j] = ok ? __builtin_amdgcn_exp2f(s[j] - mn) : 0.0f;
        float sum = p[j];
        for (int d = 32; d >= 1; d >>= 1) sum += xor_shfl(sum, d);
        l_run[j] = l_run[j] * al + sum;
        m_run[j] = mn;
        ac[j][0] *= al;
        ac[j][1] *= al;
      }
    }
    const int n = (a.n_tokens - t0) < kWave ? (a.n_tokens - t0) : kWave;
    for (int i = 0; i < n; ++i) {
      const uint16_t* vr = vbase + (size_t)((t0 + i) % cap) * kD;
      const uint32_t w = *reinterpret_cast<const uint32_t*>(vr + 2 * lane);
      const float v0 = widen(w & 0xffffu, a.is_bf16);
      const float v1 = widen(w >> 16, a.is_bf16);
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        if (j < a.G) {
          const float pj = __shfl(p[j], i, kWave);
          ac[j][0] = __builtin_fmaf(pj, v0, ac[j][0]);
          ac[j][1] = __builtin_fmaf(pj, v1, ac[j][1]);
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    if (j < a.G) {
      accw[j * kD + 2 * lane] = ac[j][0];
      accw[j * kD + 2 * lane + 1] = ac[j][1];
      if (lane == 0) {
        ml[2 * j] = m_run[j];
        ml[2 * j + 1] = l_run[j];
      }
    }
  }
}

constexpr int kWavesPerBlock = 4;

__global__ void __launch_bounds__(kWave * kWavesPerBlock)
attn_kernel(AttnLaunch a) {
  __shared__ float qs[16][kD];
  const int h = blockIdx.y, b = blockIdx.z;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
  const int split = blockIdx.x * kWavesPerBlock + wave;
  const size_t unit = (size_t)b * a.H + h;
  const size_t part = unit * (a.n_split + 1) + split;
  float* ml = a.ws_ml + part * a.G * 2;
  float* accw = a.ws_acc + part * a.G * kD;

  // Only the workgroup holding the residual split needs plain queries; the
  // window holds unrotated tokens.
  const int last_wg = a.n_split / kWavesPerBlock;
  const bool has_resid = (int)blockIdx.x == last_wg;
  const bool quarot = a.family == RQ_QUAROT;
  if (has_resid && quarot) {
    load_queries(a, b, h, false, qs);
    if (split == a.n_split) residual_split(a, b, h, qs, ml, accw);
    __syncthreads();
    load_queries(a, b, h, true, qs);
  } else {
    load_queries(a, b, h, quarot, qs);
    if (split == a.n_split) residual_split(a, b, h, qs, ml, accw);
  }
  if (split >= a.n_split) return;

  const int r = lane >> 4, col = lane & 15;
  // B operand of QK: column j = col, k-slots of quarter r, K-block kb:
  // channels 32r + (4kb + k') and 32r + 16 + (4kb + k'), k' = 0..3.
  h8 qb[4];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    uint32_t x[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int c0 = 32 * r + 4 * kb + kk;
      const h2 v = {(_Float16)qs[col][c0], (_Float16)qs[col][c0 + 16]};
      x[kk] = as_u32(v);
    }
    qb[kb] = make_h8(x[0], x[1], x[2], x[3]);
  }

  const int bk = a.tab.bits[h][0], bv = a.tab.bits[h][1];
  const int nblk_cap = a.cap / kChunk;
  const int per_blk = quarot ? kMetaBlockTok : kMetaBlockKivi;
  KCtx kc;
  kc.region = reinterpret_cast<const uint32_t*>(a.codes + a.tab.code_off[h][0]) +
              (size_t)b * a.cap * 4 * bk;
  kc.meta = a.meta + (((size_t)h * 2 + 0) * a.B + b) * nblk_cap * per_blk;
  kc.r = r;
  kc.m = col;
  VCtx vc;
  vc.region = reinterpret_cast<const uint32_t*>(a.codes + a.tab.code_off[h][1]) +
              (size_t)b * nblk_cap * kD * bv;
  vc.meta = a.meta + (((size_t)h * 2 + 1) * a.B + b) * nblk_cap * per_blk;
  vc.r = r;
  vc.n = col;

  f4 acc[8];
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) acc[nt] = (f4){0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.0f;

  const int nblk = a.nq / kChunk;
  const int blk_lo = split * a.blk_per_split;
  int blk_hi = blk_lo + a.blk_per_split;
  if (blk_hi > nblk) blk_hi = nblk;

  for (int blk = blk_lo; blk < blk_hi; ++blk) {
    f4 S0, S1;
    if (quarot) {
      RQ_DISPATCH8(bk, qk_quarot, kc, blk, qb, S0, S1)
    } else {
      RQ_DISPATCH8(bk, qk_kivi, kc, blk, qb, S0, S1)
    }
    // online softmax for column col (query j = col), tokens 4r+i, 16+4r+i
    float mx = S0[0];
#pragma unroll
    for (int i = 0; i < 4; ++i) mx = __builtin_fmaxf(mx, __builtin_fmaxf(S0[i], S1[i]));
    mx = __builtin_fmaxf(mx, xor_shfl(mx, 16));
    mx = __builtin_fmaxf(mx, xor_shfl(mx, 32));
    const float mnew = __builtin_fmaxf(m_run, mx);
    const float alpha = __builtin_amdgcn_exp2f(m_run - mnew);
    m_run = mnew;
    float p0[4], p1[4], psum = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      p0[i] = __builtin_amdgcn_exp2f(S0[i] - mnew);
      p1[i] = __builtin_amdgcn_exp2f(S1[i] - mnew);
      psum += p0[i] + p1[i];
    }
    l_run = l_run * alpha + psum;
    // rescale accumulator rows 4r + i by alpha of column 4r + i
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float ar = __shfl(alpha, 4 * r + i, kWave);
#pragma unroll
      for (int nt = 0; nt < 8; ++nt) acc[nt][i] *= ar;
    }
    uint32_t pp[4];
    if (quarot) {
      const u4 sv = *reinterpret_cast<const u4*>(vc.meta + (size_t)blk * kMetaBlockTok +
                                                 r * 16);
      const uint32_t ss[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const h2 s = as_h2(ss[i]);
        const h2 pv = {(_Float16)(p0[i] * (float)s.x), (_Float16)(p1[i] * (float)s.y)};
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
    if (quarot) {
      RQ_DISPATCH8(bv, pv_quarot, vc, blk, P, acc)
    } else {
      RQ_DISPATCH8(bv, pv_kivi, vc, blk, P, acc)
    }
  }
  // partial sums of l over the 4 lane quarters
  l_run += xor_shfl(l_run, 16);
  l_run += xor_shfl(l_run, 32);
  if (r == 0 && col < a.G) {
    ml[2 * col] = m_run;
    ml[2 * col + 1] = l_run;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int j = 4 * r + i;
    if (j < a.G) {
#pragma unroll
      for (int nt = 0; nt < 8; ++nt) accw[j * kD + 16 * nt + col] = acc[nt][i];
    }
  }
}

__global__ void __launch_bounds__(kD)
combine_kernel(AttnLaunch a) {
  __shared__ float o[kD];
  const int bq = blockIdx.x;               // b * Hq + hq
  const int b = bq / (a.H * a.G), hq = bq % (a.H * a.G);
  const int h = hq / a.G, j = hq % a.G;
  const int c = threadIdx.x;
  const size_t unit = (size_t)b * a.H + h;
  const int ns = a.n_split + 1;
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) {
    const float* ml = a.ws_ml + ((unit * ns + s) * a.G + j) * 2;
    M = __builtin_fmaxf(M, ml[0]);
  }
  float num = 0.0f, den = 0.0f, numr = 0.0f;
  for (int s = 0; s < ns; ++s) {
    const float* ml = a.ws_ml + ((unit * ns + s) * a.G + j) * 2;
    const float w = (ml[1] > 0.0f) ? __builtin_amdgcn_exp2f(ml[0] - M) : 0.0f;
    const float v = a.ws_acc[((unit * ns + s) * a.G + j) * kD + c];
    if (s == a.n_split) numr += w * v; else num += w * v;
    den += w * ml[1];
  }
  float res = num;
  if (a.family == RQ_QUAROT) {
    // quantized part is in the rotated domain: out = (1/sqrt(128)) H acc
    o[c] = num;
    __syncthreads();
    for (int hh = 1; hh < kD; hh *= 2) {
      float x = 0.0f;
      const int partner = c ^ hh;
      x = (c & hh) ? (o[partner] - o[c]) : (o[c] + o[partner]);
      __syncthreads();
      o[c] = x;
      __syncthreads();
    }
    res = o[c] * kInvSqrtD;
  }
  a.out[(size_t)bq * kD + c] = (res + numr) / den;
}

}  // namespace

hipError_t launch_attention(const AttnLaunch& a, hipStream_t s) {
  dim3 grid((a.n_split + kWavesPerBlock) / kWavesPerBlock, a.H, a.B);
  hipLaunchKernelGGL(attn_kernel, grid, dim3(kWave * kWavesPerBlock), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(combine_kernel, dim3(a.B * a.H * a.G), dim3(kD), 0, s, a);
  return hipGetLastError();
}

}  // namespace rq
