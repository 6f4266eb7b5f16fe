// Decode attention: launch glue and the kernel that merges the partials of
// the streaming workgroups (the streaming kernel itself is in
// rq_attn_impl.h, one translation unit per variant).
#include "rq_attn_impl.h"

namespace rq {

hipError_t launch_attn_kivi_n1_b4(const AttnLaunch&, size_t, hipStream_t);
hipError_t launch_attn_kivi_n1_b8(const AttnLaunch&, size_t, hipStream_t);
hipError_t launch_attn_kivi_n2_b4(const AttnLaunch&, size_t, hipStream_t);
hipError_t launch_attn_kivi_n2_b8(const AttnLaunch&, size_t, hipStream_t);
hipError_t launch_attn_kivi_n4_b4(const AttnLaunch&, size_t, hipStream_t);
hipError_t launch_attn_kivi_n4_b8(const AttnLaunch&, size_t, hipStream_t);
hipError_t launch_attn_quarot_b4(const AttnLaunch&, size_t, hipStream_t);
hipError_t launch_attn_quarot_b8(const AttnLaunch&, size_t, hipStream_t);

namespace {

// Merge the partials of one (batch, kv-head) unit: one workgroup per unit.
// It first attends to the unit's 16-bit residual window (original domain):
// run after the streaming kernel, its few dependent loads see an idle memory
// system.  Slots 0 .. n_wg-1 hold the quantized blocks (QuaRot: rotated
// domain), the residual partial is kept in LDS as slot n_wg.
__global__ void __launch_bounds__(kThreads)
combine_kernel(AttnLaunch a) {
  extern __shared__ u4 cdyn[];
  const int unit = blockIdx.x, tid = threadIdx.x;
  const int b = unit / a.H, h = unit % a.H;
  const int G = a.G;
  const bool quarot = a.family == RQ_QUAROT;
  const int ns = a.n_wg + 1;
  uint8_t* base = reinterpret_cast<uint8_t*>(cdyn);
  uint16_t* stage = reinterpret_cast<uint16_t*>(base);           // window staging
  float* rot = reinterpret_cast<float*>(base);                   // reuses the staging
  float (*qs)[kD] = reinterpret_cast<float (*)[kD]>(base + kResLds);
  float* resid = reinterpret_cast<float*>(base + kResLds + 16 * kD * sizeof(float));
  float* wgt = resid + 16 * (2 + kD);
  float* lsum = wgt + ns * G;
  __shared__ float inv_den[16];
  // (max, sum) of the streamed slots
  for (int e = tid; e < a.n_wg * G; e += kThreads) {
    const float* src = part_ptr(a, unit, e / G) + (e % G) * (2 + kD);
    wgt[e] = src[0];
    lsum[e] = src[1];
  }
  // the residual window, into LDS
  const u4 qpiece = query_piece(a, b, h);
  store_queries(a, qpiece, false, qs);
  residual_slot(a, b, h, qs, stage, resid);
  __syncthreads();
  for (int e = tid; e < G; e += kThreads) {
    wgt[a.n_wg * G + e] = resid[e * (2 + kD)];
    lsum[a.n_wg * G + e] = resid[e * (2 + kD) + 1];
  }
  __syncthreads();
  if (tid < G) {
    float M = -INFINITY;
    for (int sl = 0; sl < ns; ++sl)
      if (lsum[sl * G + tid] > 0.0f) M = __builtin_fmaxf(M, wgt[sl * G + tid]);
    float den = 0.0f;
    for (int sl = 0; sl < ns; ++sl) {
      const float m = wgt[sl * G + tid];
      const float f = lsum[sl * G + tid] > 0.0f ? __builtin_amdgcn_exp2f(m - M) : 0.0f;
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
    for (int sl = 0; sl < a.n_wg; ++sl) num = __builtin_fmaf(wgt[sl * G + j], src[sl * stride], num);
    tailv[n_e] = wgt[a.n_wg * G + j] * resid[j * (2 + kD) + 2 + cc];
    rot[e] = num;
  }
  __syncthreads();
  if (quarot) {
    for (int hh = 1; hh < kD; hh *= 2) {
      for (int e = tid; e < G * (kD / 2); e += kThreads) {
        const int j = e / (kD / 2), i = e % (kD / 2);
        const int base2 = (i / hh) * 2 * hh + (i % hh);
        const float x = rot[j * kD + base2], y = rot[j * kD + base2 + hh];
        rot[j * kD + base2] = x + y;
        rot[j * kD + base2 + hh] = x - y;
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

size_t attention_area_bytes(int G, int slot_bytes, int maxb) {
  const size_t merge = (size_t)kWaves * G * (2 + kD) * sizeof(float);
  const size_t slots = (size_t)kWaves * attn_depth(maxb) * slot_bytes;
  size_t m = merge > slots ? merge : slots;
  return (m + 15) / 16 * 16;
}

size_t attention_lds_bytes(int G, int slot_bytes, int maxb) {
  return attention_area_bytes(G, slot_bytes, maxb) + (size_t)16 * kD * sizeof(float) +
         (size_t)16 * kD * sizeof(uint16_t);
}

size_t combine_lds_bytes(int G, int n_wg) {
  return kResLds + (size_t)16 * kD * sizeof(float) + (size_t)16 * (2 + kD) * sizeof(float) +
         (size_t)2 * (n_wg + 1) * G * sizeof(float);
}

hipError_t launch_attention(const AttnLaunch& a, hipStream_t s) {
  int maxb = 1;
  for (int h = 0; h < a.H; ++h)
    for (int k = 0; k < 2; ++k) maxb = a.tab.bits[h][k] > maxb ? a.tab.bits[h][k] : maxb;
  const size_t lds = attention_lds_bytes(a.G, a.slot_bytes, maxb);
  const bool wide = maxb > 4;
  hipError_t e;
  if (a.n_wg == 0)
    e = hipSuccess;   // nothing quantized yet: the window is all there is
  else if (a.family == RQ_QUAROT)
    e = (wide ? launch_attn_quarot_b8 : launch_attn_quarot_b4)(a, lds, s);
  else if (a.GP <= 4)
    e = (wide ? launch_attn_kivi_n1_b8 : launch_attn_kivi_n1_b4)(a, lds, s);
  else if (a.GP == 8)
    e = (wide ? launch_attn_kivi_n2_b8 : launch_attn_kivi_n2_b4)(a, lds, s);
  else
    e = (wide ? launch_attn_kivi_n4_b8 : launch_attn_kivi_n4_b4)(a, lds, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(combine_kernel, dim3(a.B * a.H), dim3(kThreads),
                     combine_lds_bytes(a.G, a.n_wg), s, a);
  return hipGetLastError();
}

}  // namespace rq
