// TurboQuant-style quantize + pack (Sec. 2; Sec. 3.1 and Table 6 for the
// codebook): per token, y = R x with the (layer, kv-head) rotation R, the
// norm n = |x| (fp16), and per coordinate the code of t = y sqrt(128) / n
// among the b-bit Lloyd-Max thresholds of N(0,1).
//
// A workgroup serves one kv-head: R sits in LDS (rows padded to 272 bytes)
// and its four waves loop over that head's blocks (block, batch entry,
// K|V), the next block's rows already loading into registers.  A block's
// 16-bit rows are loaded straight into matrix-core operands:
//   keys   D[coord][token] = R . X^T   (the chunk of a token is 32 coords)
//   values D[token][coord] = X . R^T   (the chunk of a coord is 32 tokens)
// on v_mfma_f32_16x16x32 (bf16 inputs; fp16 inputs with R converted to
// fp16, exact for the entries of magnitude 2^-17 and above, about one entry
// of a Haar matrix rounding to the fp16 subnormal grid, by at most 2^-25).
// Norms are summed in fp64 from the same registers.  Codes count the
// positive thresholds below |t| (the codebook is symmetric, with the middle
// threshold at 0).  Codes go through a small LDS buffer from which each
// lane packs whole chunks: three-bit codes as quarters of a chunk already
// in stream order, other widths as bytes.
#include "rq_device.h"
#include "rq_internal.h"
#include "rq_ring.h"

namespace rq {

namespace {

constexpr int kWave = 64;
constexpr int kTWaves = 4;       // waves per workgroup
constexpr int kTOcc = 3;         // workgroups per CU
constexpr int kRRow = 136;       // 16-bit entries per LDS row of R (272 B)
constexpr int kUnitW = 9;        // dwords per chunk of code bytes in LDS (36 B)
constexpr float kSqrtD = 11.313708498984761f;   // fp32 nearest to sqrt(128)

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

template <int BF16>
__device__ __forceinline__ f4 mma(u4 a, u4 b, f4 c) {
  if constexpr (BF16)
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, a),
                                                   __builtin_bit_cast(bf8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, a),
                                                  __builtin_bit_cast(h8, b), c, 0, 0, 0);
}

template <int BF16>
__device__ __forceinline__ float wid(uint32_t w16) {
  if (BF16) return __uint_as_float(w16 << 16);
  return (float)__builtin_bit_cast(_Float16, (uint16_t)w16);
}

// bf16 -> fp16 bit pattern: exact for |r| >= 2^-17 (the 8 significant bits
// of a bf16 value fit the fp16 grid there); smaller entries round to the
// fp16 subnormal grid (spacing 2^-24)
__device__ __forceinline__ uint32_t bf16_to_f16(uint32_t b) {
  return __builtin_bit_cast(uint16_t, (_Float16)__uint_as_float(b << 16));
}

struct TBlock {
  int blk, b, kind;
};

__device__ __forceinline__ TBlock turbo_block(const QuantLaunch& a, int it) {
  TBlock id;
  id.blk = a.blk0 + it % a.nblk;
  const int z = it / a.nblk;
  id.b = z >> 1;
  id.kind = z & 1;
  return id;
}

__device__ __forceinline__ const uint16_t* row_src(const QuantLaunch& a, int b, int h,
                                                   int kind, int t) {
  if (t >= a.n_past) {
    const uint16_t* base = kind ? a.v : a.k;
    return base + ((size_t)(b * a.H + h) * a.n_new + (t - a.n_past)) * kD;
  }
  const int cap = a.R + kChunk;
  return a.resid + ((((size_t)b * a.H + h) * 2 + kind) * cap + (t % cap)) * kD;
}

// Operand registers of a block: x[4 tt + ks] holds, in lane l, 16-bit
// channels 32 ks + 8 (l / 16) .. + 7 of token 16 tt + l % 16.
__device__ __forceinline__ void load_x(const QuantLaunch& a, int h, const TBlock& id,
                                       u4 x[8], int lane) {
  const int t0 = id.blk * kChunk;
  const int g = lane >> 4, j = lane & 15;
  if (t0 >= a.n_past) {
    const RQ_GLOBAL u4* src = gptr(reinterpret_cast<const u4*>(
        (id.kind ? a.v : a.k) +
        ((size_t)(id.b * a.H + h) * a.n_new + (t0 - a.n_past)) * kD));
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) x[4 * tt + ks] = src[(16 * tt + j) * 16 + 4 * ks + g];
  } else {
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const RQ_GLOBAL u4* row = gptr(reinterpret_cast<const u4*>(
          row_src(a, id.b, h, id.kind, t0 + 16 * tt + j)));
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) x[4 * tt + ks] = row[4 * ks + g];
    }
  }
}

// R operand of coordinate tile ct, k-step ks: lane l holds R[16 ct + l % 16]
// [32 ks + 8 (l / 16) .. + 7] (the A operand of R . X^T and the B operand of
// X . R^T have the same lane layout).
__device__ __forceinline__ u4 r_op(const uint16_t* Rs, int ct, int ks, int lane) {
  return *reinterpret_cast<const u4*>(
      &Rs[(16 * ct + (lane & 15)) * kRRow + 32 * ks + 8 * (lane >> 4)]);
}

// Code of t: the number of thresholds below t.  th[] holds the P positive
// thresholds (ascending); the L - 1 thresholds are -th reversed, 0, th.
// cnt = #{j : th[j] < |t|}, found by bisection for b = 3 and 4 (the same
// count: the thresholds are sorted).
template <int B>
__device__ __forceinline__ uint32_t turbo_code(float t, const float* th) {
  constexpr int L = 1 << B, P = L / 2 - 1;
  const float m = __builtin_fabsf(t);
  uint32_t cnt = 0;
  if constexpr (B == 3) {
    const bool c1 = th[1] < m;
    cnt = (c1 ? 2u : 0u) + ((c1 ? th[2] : th[0]) < m ? 1u : 0u);
  } else if constexpr (B == 4) {
    const bool c1 = th[3] < m;
    const bool c2 = (c1 ? th[5] : th[1]) < m;
    const float t3 = c1 ? (c2 ? th[6] : th[4]) : (c2 ? th[2] : th[0]);
    cnt = (c1 ? 4u : 0u) + (c2 ? 2u : 0u) + (t3 < m ? 1u : 0u);
  } else {
#pragma unroll
    for (int j = 0; j < P; ++j) cnt += th[j] < m ? 1u : 0u;
  }
  return t > 0.0f ? (uint32_t)(L / 2) + cnt : (uint32_t)(L / 2 - 1) - cnt;
}

// Three-bit codes: in both operand layouts a lane holds quarter g = lane /
// 16 of one chunk (codes 4g + i and 16 + 4g + i, i = 0..3), which it
// assembles as the chunk's stream bits 24g .. 24g + 23 and stages as one
// dword (kQ3W dwords per chunk, padded against bank conflicts); the pack
// step joins a chunk's four quarters into its three words.
constexpr int kQ3W = 5;

__device__ __forceinline__ uint32_t bytes4(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3) {
  return c0 | (c1 << 8) | (c2 << 16) | (c3 << 24);
}

template <int BF16, int B>
__device__ __forceinline__ void turbo_block_codes(const QuantLaunch& a, const uint16_t* Rs,
                                                  uint32_t* cbuf, int h, const TBlock& id,
                                                  const u4 x[8], int lane) {
  constexpr int L = 1 << B, P = L / 2 - 1;
  const int g = lane >> 4, j = lane & 15;
  const int t0 = id.blk * kChunk;
  float th[P > 0 ? P : 1];
  {
    const RQ_GLOBAL float* tp = gptr(a.cb + (B - 1) * 512 + L / 2);
#pragma unroll
    for (int k = 0; k < P; ++k) th[k] = tp[k];
  }
  // norms of tokens 16 tt + j: fp64 sum of squares over the lane's 32
  // channels, then over the four lanes holding the other channels
  float f[2];
  uint32_t n16[2];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    double s = 0.0;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const u4 w = x[4 * tt + ks];
      const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double lo = (double)wid<BF16>(ww[e] & 0xffffu);
        const double hi = (double)wid<BF16>(ww[e] >> 16);
        s = __builtin_fma(lo, lo, s);
        s = __builtin_fma(hi, hi, s);
      }
    }
    s += __shfl_xor(s, 16, kWave);
    s += __shfl_xor(s, 32, kWave);
    n16[tt] = f16_sat((float)__builtin_sqrt(s));
    const float nf = f16_to_f32((uint16_t)n16[tt]);
    f[tt] = nf != 0.0f ? kSqrtD / nf : 0.0f;
  }
  // metadata: token 16 tt + j at pair position 2 j + tt
  if (g == 0) {
    const int nblk_cap = a.cap / kChunk;
    RQ_GLOBAL uint32_t* m = gptr(reinterpret_cast<uint32_t*>(
        a.meta + ((((size_t)h * 2 + id.kind) * a.B + id.b) * nblk_cap + id.blk) *
                     kMetaBlockTok));
    m[j] = n16[0] | (n16[1] << 16);
  }
  if (id.kind == 0) {
    // keys: chunk q of token 16 tt + j = coordinate tiles 2q, 2q + 1
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      f4 d[2][2];
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) d[c][tt] = (f4){0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const u4 r0 = r_op(Rs, 2 * q, ks, lane), r1 = r_op(Rs, 2 * q + 1, ks, lane);
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
          d[0][tt] = mma<BF16>(r0, x[4 * tt + ks], d[0][tt]);
          d[1][tt] = mma<BF16>(r1, x[4 * tt + ks], d[1][tt]);
        }
      }
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        // lane: token 16 tt + j, coords 32q + 16c + 4g + i -> code 16c + 4g + i
        if constexpr (B == 3) {
          uint32_t qb = 0;
#pragma unroll
          for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              qb |= turbo_code<3>(d[c][tt][i] * f[tt], th) << (12 * c + 3 * i);
          cbuf[((16 * tt + j) * 4 + q) * kQ3W + g] = qb;
        } else {
          uint32_t* u = cbuf + ((16 * tt + j) * 4 + q) * kUnitW;
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const f4 y = d[c][tt];
            u[4 * c + g] = bytes4(turbo_code<B>(y[0] * f[tt], th), turbo_code<B>(y[1] * f[tt], th),
                                  turbo_code<B>(y[2] * f[tt], th), turbo_code<B>(y[3] * f[tt], th));
          }
        }
      }
    }
  } else {
    // values: chunk of coord 16 ct + j = its 32 tokens; rows 16 tt + 4g + i
    float fr[2][4];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) fr[tt][i] = __shfl(f[tt], 4 * g + i, kWave);
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) {
      f4 d[2] = {(f4){0.0f, 0.0f, 0.0f, 0.0f}, (f4){0.0f, 0.0f, 0.0f, 0.0f}};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const u4 r = r_op(Rs, ct, ks, lane);
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) d[tt] = mma<BF16>(x[4 * tt + ks], r, d[tt]);
      }
      if constexpr (B == 3) {
        // lane: coord 16 ct + j, tokens 16 tt + 4g + i -> code 16 tt + 4g + i
        uint32_t qb = 0;
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            qb |= turbo_code<3>(d[tt][i] * fr[tt][i], th) << (12 * tt + 3 * i);
        cbuf[(16 * ct + j) * kQ3W + g] = qb;
      } else {
        uint32_t* u = cbuf + (16 * ct + j) * kUnitW;
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
          const f4 y = d[tt];
          u[4 * tt + g] = bytes4(turbo_code<B>(y[0] * fr[tt][0], th), turbo_code<B>(y[1] * fr[tt][1], th),
                                 turbo_code<B>(y[2] * fr[tt][2], th), turbo_code<B>(y[3] * fr[tt][3], th));
        }
      }
    }
  }
  __builtin_amdgcn_wave_barrier();
  // pack: units lane and lane + 64 (keys: unit = token * 4 + q; values:
  // unit = coord)
  const int nblk_cap = a.cap / kChunk;
  uint32_t* region = reinterpret_cast<uint32_t*>(a.codes + a.tab.code_off[h][id.kind]);
  uint32_t* base = id.kind == 0 ? region + ((size_t)id.b * a.cap + t0) * 4 * B
                                : region + ((size_t)id.b * nblk_cap + id.blk) * kD * B;
  if constexpr (B == 3) {
#pragma unroll
    for (int rep = 0; rep < 2; ++rep) {
      const int unit = lane + rep * kWave;
      const uint32_t* src = cbuf + unit * kQ3W;
      const uint32_t q0 = src[0], q1 = src[1], q2 = src[2], q3 = src[3];
      // words 0..2 = stream bits 0..31, 32..63, 64..95
      RQ_GLOBAL uint32_t* dst = gptr(base + (size_t)unit * 3);
      __builtin_nontemporal_store(q0 | (q1 << 24), dst);
      __builtin_nontemporal_store(__builtin_amdgcn_alignbit(q2, q1 << 8, 16), dst + 1);
      __builtin_nontemporal_store(__builtin_amdgcn_alignbit(q3, q2 << 8, 24), dst + 2);
    }
    __builtin_amdgcn_wave_barrier();
    return;
  }
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    const int unit = lane + rep * kWave;
    const uint32_t* src = cbuf + unit * kUnitW;
    uint32_t c[8], w[B];
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = src[i];
    pack_chunk<B>(c, w);
    RQ_GLOBAL uint32_t* dst = gptr(base + (size_t)unit * B);
#pragma unroll
    for (int i = 0; i < B; ++i) __builtin_nontemporal_store(w[i], dst + i);
  }
  __builtin_amdgcn_wave_barrier();
}

template <int BF16>
__device__ __forceinline__ void turbo_dispatch(const QuantLaunch& a, const uint16_t* Rs,
                                               uint32_t* cbuf, int h, const TBlock& id,
                                               const u4 x[8], int lane) {
  switch (kernarg_byte(&a.tab.bits[0][0], 2 * h + id.kind)) {
    case 1: turbo_block_codes<BF16, 1>(a, Rs, cbuf, h, id, x, lane); break;
    case 2: turbo_block_codes<BF16, 2>(a, Rs, cbuf, h, id, x, lane); break;
    case 3: turbo_block_codes<BF16, 3>(a, Rs, cbuf, h, id, x, lane); break;
    case 4: turbo_block_codes<BF16, 4>(a, Rs, cbuf, h, id, x, lane); break;
    case 5: turbo_block_codes<BF16, 5>(a, Rs, cbuf, h, id, x, lane); break;
    case 6: turbo_block_codes<BF16, 6>(a, Rs, cbuf, h, id, x, lane); break;
    case 7: turbo_block_codes<BF16, 7>(a, Rs, cbuf, h, id, x, lane); break;
    case 8: turbo_block_codes<BF16, 8>(a, Rs, cbuf, h, id, x, lane); break;
    default: break;
  }
}

// grid (workgroups per head, kv-heads)
template <int BF16>
__global__ void __launch_bounds__(kTWaves * kWave, kTOcc)
turbo_quant_kernel(QuantLaunch a) {
  __shared__ uint16_t Rs[kD * kRRow];
  __shared__ uint32_t cbuf_all[kTWaves][kD * kUnitW];
  const int h = blockIdx.y;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & (kWave - 1);
  {
    // R of this head, 16-byte pieces (row i / 16, piece i % 16)
    const RQ_GLOBAL u4* src = gptr(reinterpret_cast<const u4*>(a.rot + (size_t)h * kD * kD));
    for (int i = threadIdx.x; i < kD * 16; i += kTWaves * kWave) {
      u4 v = src[i];
      if (!BF16) {
        v.x = bf16_to_f16(v.x & 0xffffu) | (bf16_to_f16(v.x >> 16) << 16);
        v.y = bf16_to_f16(v.y & 0xffffu) | (bf16_to_f16(v.y >> 16) << 16);
        v.z = bf16_to_f16(v.z & 0xffffu) | (bf16_to_f16(v.z >> 16) << 16);
        v.w = bf16_to_f16(v.w & 0xffffu) | (bf16_to_f16(v.w >> 16) << 16);
      }
      *reinterpret_cast<u4*>(&Rs[(i >> 4) * kRRow + (i & 15) * 8]) = v;
    }
  }
  __syncthreads();
  uint32_t* cbuf = cbuf_all[wave];
  const int per_head = a.nblk * a.B * 2;
  const int stride = gridDim.x * kTWaves;
  int it = blockIdx.x * kTWaves + wave;
  if (it < per_head) {
    u4 nx[8];
    load_x(a, h, turbo_block(a, it), nx, lane);
    for (; it < per_head; it += stride) {
      const TBlock id = turbo_block(a, it);
      u4 x[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = nx[i];
      if (it + stride < per_head) load_x(a, h, turbo_block(a, it + stride), nx, lane);
      turbo_dispatch<BF16>(a, Rs, cbuf, h, id, x, lane);
    }
  }
  // the window rows of the append, after the blocks (fewer live registers)
  if (a.ring_fused)
    copy_window(a.ring, (blockIdx.y * gridDim.x + blockIdx.x) * kTWaves + wave,
                gridDim.x * gridDim.y * kTWaves, lane);
}

}  // namespace

hipError_t launch_quantize_turbo(const QuantLaunch& a, hipStream_t s) {
  if (a.nblk <= 0) return hipSuccess;
  const long per_head = (long)a.nblk * a.B * 2;
  long per = ((long)(a.n_cu > 0 ? a.n_cu : 256) * kTOcc + a.H - 1) / a.H;
  const long need = (per_head + kTWaves - 1) / kTWaves;
  if (per > need) per = need;
  if (per < 1) per = 1;
  dim3 grid((unsigned)per, a.H), block(kTWaves * kWave);
  if (a.is_bf16)
    hipLaunchKernelGGL(turbo_quant_kernel<1>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(turbo_quant_kernel<0>, grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace rq
