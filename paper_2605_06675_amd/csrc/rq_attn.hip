// Decode attention: launch glue (the kernel is in rq_attn_impl.h, one
// translation unit per variant).
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
hipError_t launch_attn_turbo_b4(const AttnLaunch&, size_t, hipStream_t);
hipError_t launch_attn_turbo_b8(const AttnLaunch&, size_t, hipStream_t);
hipError_t launch_attn_kivirtn_b4(const AttnLaunch&, size_t, hipStream_t);
hipError_t launch_attn_kivirtn_b8(const AttnLaunch&, size_t, hipStream_t);

size_t attention_area_bytes(int G, int wave_bytes, int family) {
  const size_t merge = (size_t)kWaves * G * (2 + kD) * sizeof(float);
  const size_t rings = (size_t)kWaves * wave_bytes;
  // the merging workgroup's scratch (and the rotation for TurboQuant) and
  // the window staging with its scaled query rows reuse it
  const size_t mscratch = (size_t)G * kD * sizeof(float) +
                          (family == RQ_TURBO ? (size_t)kD * kD * sizeof(uint16_t) : 0);
  const size_t window = kResLds + (size_t)16 * kD * sizeof(float);
  size_t m = merge > rings ? merge : rings;
  m = m > window ? m : window;
  m = m > mscratch ? m : mscratch;
  return (m + 15) / 16 * 16;
}

size_t attention_tail_bytes(int G, int family) {
  // TurboQuant: the rotated query rows and the K and V code tables
  return (size_t)G * kD * sizeof(uint16_t) +
         (family == RQ_TURBO ? (size_t)G * kD * sizeof(float) + 2 * kTqTabBytes : 0);
}

size_t attention_lds_bytes(int G, int wave_bytes, int family) {
  return attention_area_bytes(G, wave_bytes, family) + attention_tail_bytes(G, family);
}

hipError_t launch_attention(const AttnLaunch& a, hipStream_t s) {
  int maxb = 1;
  for (int h = 0; h < a.H; ++h)
    for (int k = 0; k < 2; ++k) maxb = a.tab.bits[h][k] > maxb ? a.tab.bits[h][k] : maxb;
  const size_t lds = attention_lds_bytes(a.G, a.wave_bytes, a.family);
  const bool wide = maxb > 4;
  hipError_t e;
  if (a.family == RQ_TURBO)
    e = (wide ? launch_attn_turbo_b8 : launch_attn_turbo_b4)(a, lds, s);
  else if (a.family == RQ_QUAROT || a.family == RQ_RTN)   // same kernel, no rotation
    e = (wide ? launch_attn_quarot_b8 : launch_attn_quarot_b4)(a, lds, s);
  else if (a.family == RQ_KIVI_RTN)
    e = (wide ? launch_attn_kivirtn_b8 : launch_attn_kivirtn_b4)(a, lds, s);
  else if (a.GP <= 4)
    e = (wide ? launch_attn_kivi_n1_b8 : launch_attn_kivi_n1_b4)(a, lds, s);
  else if (a.GP == 8)
    e = (wide ? launch_attn_kivi_n2_b8 : launch_attn_kivi_n2_b4)(a, lds, s);
  else
    e = (wide ? launch_attn_kivi_n4_b8 : launch_attn_kivi_n4_b4)(a, lds, s);
  return e;
}

}  // namespace rq
