// C-ABI entry points: validation, cache layout, launch set-up.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "rq_host.h"
#include "rq_internal.h"

namespace {

thread_local std::string g_err;

rq_status fail(rq_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

rq_status ok() {
  g_err.clear();
  return RQ_OK;
}

rq_status hip_fail(hipError_t e, const char* what) {
  return fail(RQ_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

int n_quantized(int T, int R) {
  const int x = T - R;
  return x <= 0 ? 0 : (x / rq::kChunk) * rq::kChunk;
}

// metadata bytes of one block of K plus one of V
int meta_pair_bytes(const rq_cache* c) {
  return rq::meta_block_bytes(c->family, 0) + rq::meta_block_bytes(c->family, 1);
}

rq_status check_cache(const rq_cache* c) {
  if (!c) return fail(RQ_EINVAL, "cache descriptor is NULL");
  if (c->family != RQ_KIVI && c->family != RQ_QUAROT && c->family != RQ_TURBO &&
      c->family != RQ_RTN && c->family != RQ_KIVI_RTN)
    return fail(RQ_EINVAL, "unknown family %d", c->family);
  if (c->family == RQ_TURBO && (!c->rotation || !c->codebook))
    return fail(RQ_EINVAL, "TurboQuant needs the rotation and codebook pointers");
  if (c->dtype != RQ_F16 && c->dtype != RQ_BF16)
    return fail(RQ_EINVAL, "unknown dtype %d", c->dtype);
  if (c->head_dim != rq::kD)
    return fail(RQ_EUNSUPPORTED, "head_dim %d (only 128 is supported)", c->head_dim);
  if (c->n_layers < 1 || c->batch < 1)
    return fail(RQ_EINVAL, "n_layers and batch must be >= 1");
  if (c->n_kv_heads < 1 || c->n_kv_heads > RQ_MAX_KV_HEADS)
    return fail(RQ_EINVAL, "n_kv_heads %d outside 1..%d", c->n_kv_heads,
                RQ_MAX_KV_HEADS);
  if (c->n_q_heads < c->n_kv_heads || c->n_q_heads % c->n_kv_heads)
    return fail(RQ_EINVAL, "n_q_heads %d is not a multiple of n_kv_heads %d",
                c->n_q_heads, c->n_kv_heads);
  if (c->n_q_heads / c->n_kv_heads > 16)
    return fail(RQ_EUNSUPPORTED, "more than 16 query heads per kv-head");
  if (c->capacity < rq::kChunk || c->capacity % rq::kChunk)
    return fail(RQ_EINVAL, "capacity %d must be a positive multiple of 32",
                c->capacity);
  if (c->residual < 0) return fail(RQ_EINVAL, "residual window must be >= 0");
  if (!c->bits) return fail(RQ_EINVAL, "bit table is NULL");
  for (int i = 0; i < c->n_layers * c->n_kv_heads * 2; ++i) {
    const int b = c->bits[i];
    // symmetric quantizers need two bits or more: QuaRot and RTN on both
    // sides, the values (odd entries) of KIVI_RTN
    const bool sym = c->family == RQ_QUAROT || c->family == RQ_RTN ||
                     (c->family == RQ_KIVI_RTN && (i & 1));
    const int lo = sym ? 2 : 1;
    if (b < lo || b > 8)
      return fail(RQ_EINVAL, "bit table entry %d is %d (allowed %d..8)", i, b, lo);
  }
  const double codes = (double)c->n_layers * c->n_kv_heads * 2 * c->batch *
                       c->capacity * 16.0 * 8;
  if (codes > 9.0e18) return fail(RQ_EINVAL, "cache too large");
  return RQ_OK;
}

uint64_t region_bytes(const rq_cache* c, int b) {
  return (uint64_t)c->batch * c->capacity * 16 * b;
}

uint64_t region_offset(const rq_cache* c, int layer, int head, int kind) {
  uint64_t off = 0;
  const int H = c->n_kv_heads;
  const int stop = (layer * H + head) * 2 + kind;
  for (int i = 0; i < stop; ++i) off += region_bytes(c, c->bits[i]);
  return off;
}

uint64_t meta_layer_bytes(const rq_cache* c) {
  return (uint64_t)c->n_kv_heads * c->batch * (c->capacity / rq::kChunk) *
         meta_pair_bytes(c);
}

uint64_t resid_layer_elems(const rq_cache* c) {
  return (uint64_t)c->batch * c->n_kv_heads * 2 * (c->residual + rq::kChunk) *
         rq::kD;
}

rq::LayerTable layer_table(const rq_cache* c, int layer) {
  rq::LayerTable t{};
  uint64_t off = region_offset(c, layer, 0, 0);
  for (int h = 0; h < c->n_kv_heads; ++h)
    for (int kind = 0; kind < 2; ++kind) {
      const int b = c->bits[(layer * c->n_kv_heads + h) * 2 + kind];
      t.code_off[h][kind] = off;
      t.bits[h][kind] = (uint8_t)b;
      off += region_bytes(c, b);
    }
  return t;
}

// LDS bytes a workgroup may allocate on the current device (queried once;
// 64 KiB when no device can be queried).
size_t lds_limit() {
  static size_t n = 0;
  if (n == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) ==
            hipSuccess &&
        v > 0)
      n = (size_t)v;
    else
      n = 65536;
  }
  return n;
}

// LDS bytes of one CU (queried once; 160 KiB, the gfx950 size, when no
// device can be queried).
size_t lds_per_cu() {
  static size_t n = 0;
  if (n == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) ==
            hipSuccess &&
        v > 0)
      n = (size_t)v;
    else
      n = 163840;
  }
  return n;
}

struct SplitPlan {
  int nq, n_rw;
  int n_wg;                          // the largest nwg (grid slots per unit)
  int nwg[RQ_MAX_KV_HEADS];          // workgroups per unit of each kv-head
  int pstride;                       // partial slots per unit
};

// LDS shape of the attention kernel for one layer: the most workgroups per
// CU (three, the kernel's occupancy, down to one) whose share of the CU's
// LDS gives every wave a ring of at least two blocks of the layer's widest
// kv-head.  A share is rounded down to whole 2 KiB (an allocation granule
// coarser than 512 bytes was measured to lose the third workgroup), less
// 64 bytes for the static LDS.  False when not even one workgroup per CU
// fits.
struct AttnShape {
  int wg_per_cu, wave_bytes;
  size_t lds;
};

bool attn_shape(const rq_cache* c, int max_blk_bytes, AttnShape* out) {
  const int G = c->n_q_heads / c->n_kv_heads;
  const size_t tail = rq::attention_tail_bytes(G, c->family);
  for (int w = 3; w >= 1; --w) {
    size_t share = (lds_per_cu() / w) / 2048 * 2048 - 64;
    share = share < lds_limit() ? share : lds_limit();
    if (share <= tail) continue;
    const int wave = (int)((share - tail) / rq::kAttnWaves / 16 * 16);
    if (wave < 2 * max_blk_bytes) continue;
    const size_t lds = rq::attention_lds_bytes(G, wave, c->family);
    if (lds > share) continue;
    *out = AttnShape{w, wave, lds};
    return true;
  }
  return false;
}

// Compute units of the current device (queried once; 256 when no device
// can be queried, e.g. for host-only sizing calls).
int cu_count() {
  static int n = 0;
  if (n == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) ==
            hipSuccess &&
        v > 0)
      n = v;
    else
      n = 256;
  }
  return n;
}

// Merge groups of a unit's workgroups (the two-level merge starts above
// kAttnMergeFlat workgroups, in groups of kAttnGroup).
int merge_groups(int n_wg) {
  if (n_wg <= rq::kAttnMergeFlat) return 0;
  return (n_wg + rq::kAttnGroup - 1) / rq::kAttnGroup;
}

// Workgroups (four waves each) per (batch, kv-head) unit.  The grid is sized
// to one resident round with every CU busy (wg_per_cu workgroups per CU,
// three when the LDS allows), split evenly over the units, at least 4
// blocks per workgroup.  (Shares weighted by the cost of each kv-head's
// widths were measured slower on MI355X: a unit's extra workgroups land in
// the youngest residency slots, which issue last.)  The 16-bit window is
// n_rw chunks of 32 tokens, taken by the unit's first workgroups before
// their blocks.
SplitPlan plan_splits(const rq_cache* c, int layer, int n_tokens, int wg_per_cu = 3) {
  (void)layer;
  SplitPlan p{};
  p.nq = n_quantized(n_tokens, c->residual);
  p.n_rw = (n_tokens - p.nq + rq::kAttnResChunk - 1) / rq::kAttnResChunk;
  const long nblk = p.nq / rq::kChunk;
  const int H = c->n_kv_heads;
  const double budget = (double)cu_count() * wg_per_cu / ((double)c->batch * H);
  const long most = (nblk + 3) / 4;   // at least 4 blocks per workgroup
  p.n_wg = 0;
  p.pstride = 1;
  for (int h = 0; h < H; ++h) {
    long n = nblk == 0 ? 0 : (long)budget;
    if (nblk > 0 && n < 1) n = 1;
    if (n > most) n = most;
    p.nwg[h] = (int)n;
    p.n_wg = p.nwg[h] > p.n_wg ? p.nwg[h] : p.n_wg;
    const int ps = p.nwg[h] + p.n_rw + merge_groups(p.nwg[h]);
    p.pstride = ps > p.pstride ? ps : p.pstride;
  }
  return p;
}

// Counters per unit, sized for the most workgroups any call on this cache
// can use (at least 4 blocks each), so that the counter area -- zero
// between calls -- does not move: the tickets (final, one per merge group)
// in whole 128-byte lines, then one 128-byte line per claim group of
// kAttnGroup workgroups (claims contend only within their line).
int max_groups(const rq_cache* c) {
  const int max_wg = (c->capacity / rq::kChunk + 3) / 4;
  return (max_wg + rq::kAttnGroup - 1) / rq::kAttnGroup;
}
// (64-bit counters: 16 per line)
int claim_offset(const rq_cache* c) { return 16 * ((1 + max_groups(c) + 15) / 16); }
int counter_stride(const rq_cache* c) { return claim_offset(c) + 16 * max_groups(c); }

// Workspace: per-unit arrival and claim counters, padded to 256 bytes, then
// the partials [B][H][n_wg + n_rw + groups][G][2 + 128] floats.
uint64_t attn_counter_bytes(const rq_cache* c) {
  return ((uint64_t)c->batch * c->n_kv_heads * counter_stride(c) * sizeof(uint64_t) + 255) /
         256 * 256;
}

// The calls on one workspace (keyed by the address of its counters) are
// numbered 1, 2, ..; the number tags the counters the call uses, so that a
// count left by a call that did not finish is recognised as stale (0 never
// numbers a call: a zeroed counter is always stale).
uint32_t next_epoch(const void* counters) {
  static std::mutex mu;
  static std::unordered_map<const void*, uint32_t> epochs;
  std::lock_guard<std::mutex> lock(mu);
  uint32_t& e = epochs[counters];
  e = e + 1u == 0u ? 1u : e + 1u;
  return e;
}

int part_stride(const SplitPlan& p) { return p.pstride; }

uint64_t attn_ws_bytes(const rq_cache* c, const SplitPlan& p) {
  const uint64_t G = c->n_q_heads / c->n_kv_heads;
  const uint64_t parts = (uint64_t)c->batch * c->n_kv_heads * part_stride(p);
  return attn_counter_bytes(c) + parts * G * (2 + rq::kD) * sizeof(float);
}

}  // namespace

namespace rq {

uint64_t decode_counter_bytes(const rq_cache* c) { return attn_counter_bytes(c); }

rq_status decode_attention(const rq_cache* c, int32_t layer, int32_t n_tokens, const void* q,
                           float* out, float scale, void* counters, uint64_t counter_cap,
                           float* part, uint64_t part_cap, rq_stream stream,
                           const void* k_new, const void* v_new, bool launch) {
  rq_status st = check_cache(c);
  if (st != RQ_OK) return st;
  if (layer < 0 || layer >= c->n_layers)
    return fail(RQ_EINVAL, "layer %d out of range", layer);
  if (n_tokens < 1 || n_tokens > c->capacity)
    return fail(RQ_EINVAL, "n_tokens %d outside 1..%d", n_tokens, c->capacity);
  if (!q || !out || !counters || !part || !c->codes || !c->meta || !c->resid)
    return fail(RQ_EINVAL, "NULL device pointer");
  if (!std::isfinite(scale)) return fail(RQ_EINVAL, "scale is not finite");
  const rq::LayerTable tab = layer_table(c, layer);
  int max_blk = 0;
  for (int h = 0; h < c->n_kv_heads; ++h) {
    const int bb = 512 * (tab.bits[h][0] + tab.bits[h][1]) + meta_pair_bytes(c);
    max_blk = bb > max_blk ? bb : max_blk;
  }
  // each unit's K and V codes, and its K and V metadata, are read through
  // one 32-bit-addressed buffer each
  {
    const uint64_t nc = c->capacity / rq::kChunk, cap16 = (uint64_t)c->capacity * 16;
    const uint64_t mk = rq::meta_block_bytes(c->family, 0), mv = rq::meta_block_bytes(c->family, 1);
    const uint64_t B = c->batch;
    for (int h = 0; h < c->n_kv_heads; ++h) {
      const uint64_t bk = tab.bits[h][0], bv = tab.bits[h][1];
      for (uint64_t b : {(uint64_t)0, B - 1}) {
        const uint64_t codes = cap16 * ((B - b) * bk + b * bv) + cap16 * bv;
        const uint64_t meta = nc * ((B - b) * mk + b * mv) + nc * mv;
        if (codes > 0xffffffffull || meta > 0xffffffffull)
          return fail(RQ_EUNSUPPORTED,
                      "layer %d head %d: the codes of one (batch, kv-head) unit span more "
                      "than 4 GiB", layer, h);
      }
    }
  }
  AttnShape shape;
  if (!attn_shape(c, max_blk, &shape))
    return fail(RQ_EUNSUPPORTED,
                "layer %d: two %d-byte blocks per wave do not fit the LDS of a CU "
                "(K+V bit-widths of one kv-head are too wide)", layer, max_blk);
  const SplitPlan p = plan_splits(c, layer, n_tokens, shape.wg_per_cu);
  const uint64_t need_c = attn_counter_bytes(c);
  const uint64_t need_p = attn_ws_bytes(c, p) - need_c;
  if (counter_cap < need_c || part_cap < need_p)
    return fail(RQ_ESMALLWS, "workspace: counters %llu of %llu bytes, partials %llu of %llu",
                (unsigned long long)counter_cap, (unsigned long long)need_c,
                (unsigned long long)part_cap, (unsigned long long)need_p);
  const int G = c->n_q_heads / c->n_kv_heads;
  rq::AttnLaunch a{};
  a.q = static_cast<const uint16_t*>(q);
  a.codes = static_cast<const uint8_t*>(c->codes);
  a.meta = static_cast<const uint8_t*>(c->meta) + meta_layer_bytes(c) * layer;
  a.resid = static_cast<const uint16_t*>(c->resid) + resid_layer_elems(c) * layer;
  a.out = out;
  a.t_new = k_new ? n_tokens - 1 : -1;
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.resid_w = static_cast<uint16_t*>(c->resid) + resid_layer_elems(c) * layer;
  a.counters = static_cast<uint64_t*>(counters);
  a.part = part;
  a.pstride = part_stride(p);
  a.cstride = counter_stride(c);
  a.claim_off = claim_offset(c);
  a.B = c->batch;
  a.H = c->n_kv_heads;
  a.G = G;
  a.GP = 1;
  while (a.GP < G) a.GP *= 2;
  a.cap = c->capacity;
  a.R = c->residual;
  a.nq = p.nq;
  a.n_tokens = n_tokens;
  a.n_wg = p.n_wg;
  for (int h = 0; h < c->n_kv_heads; ++h) a.nwg[h] = (uint16_t)p.nwg[h];
  a.n_rw = p.n_rw;
  a.is_bf16 = c->dtype == RQ_BF16;
  a.family = c->family;
  a.qscale = scale * 1.4426950408889634f;
  if (c->family == RQ_TURBO) {
    a.rot = static_cast<const uint16_t*>(c->rotation) +
            (size_t)layer * c->n_kv_heads * rq::kD * rq::kD;
    a.cb = c->codebook;
  }
  a.tab = tab;
  a.wave_bytes = shape.wave_bytes;
  a.area_bytes = (int)rq::attention_area_bytes(G, a.wave_bytes, c->family);
  if (!launch) return ok();
  a.epoch = next_epoch(counters);
  hipError_t e = rq::launch_attention(a, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "attention launch");
  return ok();
}

rq_status set_error(rq_status code, const char* msg) { return fail(code, "%s", msg); }

}  // namespace rq

extern "C" {

int32_t rq_version(void) { return 100; }

const char* rq_last_error(void) { return g_err.c_str(); }

rq_status rq_cache_sizes(const rq_cache* c, uint64_t* codes_bytes,
                         uint64_t* meta_bytes, uint64_t* resid_bytes) {
  rq_status st = check_cache(c);
  if (st != RQ_OK) return st;
  if (codes_bytes) *codes_bytes = region_offset(c, c->n_layers, 0, 0);
  if (meta_bytes) *meta_bytes = meta_layer_bytes(c) * c->n_layers;
  if (resid_bytes)
    *resid_bytes = resid_layer_elems(c) * c->n_layers * sizeof(uint16_t);
  return ok();
}

rq_status rq_region_offset(const rq_cache* c, int32_t layer, int32_t head,
                           int32_t kind, uint64_t* offset) {
  rq_status st = check_cache(c);
  if (st != RQ_OK) return st;
  if (layer < 0 || layer >= c->n_layers || head < 0 || head >= c->n_kv_heads ||
      kind < 0 || kind > 1 || !offset)
    return fail(RQ_EINVAL, "region (%d, %d, %d) out of range", layer, head, kind);
  *offset = region_offset(c, layer, head, kind);
  return ok();
}

namespace {

// Quantize launch of the blocks that leave the residual window when n_new
// tokens (k, v: [batch][n_kv_heads][n_new][128]) follow n_past cached ones.
rq::QuantLaunch quant_launch(const rq_cache* c, int layer, int n_past, const void* k,
                             const void* v, int n_new) {
  const int nq_old = n_quantized(n_past, c->residual);
  const int nq_new = n_quantized(n_past + n_new, c->residual);
  rq::QuantLaunch q{};
  q.k = static_cast<const uint16_t*>(k);
  q.v = static_cast<const uint16_t*>(v);
  q.codes = static_cast<uint8_t*>(c->codes);
  q.meta = static_cast<uint8_t*>(c->meta) + meta_layer_bytes(c) * layer;
  q.resid = static_cast<uint16_t*>(c->resid) + resid_layer_elems(c) * layer;
  q.B = c->batch;
  q.H = c->n_kv_heads;
  q.n_new = n_new;
  q.n_past = n_past;
  q.cap = c->capacity;
  q.R = c->residual;
  q.blk0 = nq_old / rq::kChunk;
  q.nblk = (nq_new - nq_old) / rq::kChunk;
  q.is_bf16 = c->dtype == RQ_BF16;
  q.family = c->family;
  q.n_cu = cu_count();
  if (c->family == RQ_TURBO) {
    q.rot = static_cast<const uint16_t*>(c->rotation) +
            (size_t)layer * c->n_kv_heads * rq::kD * rq::kD;
    q.cb = c->codebook;
  }
  q.tab = layer_table(c, layer);
  return q;
}

}  // namespace

rq_status rq_quantize_kv(const rq_cache* c, int32_t layer, int32_t n_past,
                         const void* k, const void* v, int32_t n_new,
                         rq_stream stream) {
  rq_status st = check_cache(c);
  if (st != RQ_OK) return st;
  if (layer < 0 || layer >= c->n_layers)
    return fail(RQ_EINVAL, "layer %d out of range", layer);
  if (n_past < 0 || n_new < 1 || (int64_t)n_past + n_new > c->capacity)
    return fail(RQ_EINVAL, "tokens %d + %d exceed capacity %d", n_past, n_new,
                c->capacity);
  if (!k || !v || !c->codes || !c->meta || !c->resid)
    return fail(RQ_EINVAL, "NULL device pointer");
  const int T_new = n_past + n_new;
  const int nq_new = n_quantized(T_new, c->residual);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  rq::QuantLaunch q = quant_launch(c, layer, n_past, k, v, n_new);
  rq::RingLaunch r{};
  r.k = q.k;
  r.v = q.v;
  r.resid = q.resid;
  r.B = c->batch;
  r.H = c->n_kv_heads;
  r.n_new = n_new;
  r.n_past = n_past;
  r.R = c->residual;
  r.t_lo = nq_new > n_past ? nq_new : n_past;
  r.t_hi = T_new;
  // The quantize launch also copies the window rows unless a row it writes
  // could take the ring slot of a token a flushed block still reads there
  // (tokens [nq_old, min(nq_new, n_past)) are read from the ring): then the
  // window waits for its own launch.
  const int nq_old = n_quantized(n_past, c->residual);
  const int read_hi = nq_new < n_past ? nq_new : n_past;
  const bool reads_ring = nq_old < read_hi;
  q.ring = r;
  q.ring_fused = q.nblk > 0 && (!reads_ring || T_new - 1 - nq_old < c->residual + rq::kChunk);
  hipError_t e = rq::launch_quantize(q, s);
  if (e != hipSuccess) return hip_fail(e, "quantize launch");
  if (!q.ring_fused) {
    e = rq::launch_ring(r, s);
    if (e != hipSuccess) return hip_fail(e, "window launch");
  }
  return ok();
}

rq_status rq_decode_workspace(const rq_cache* c, int32_t n_tokens,
                              uint64_t* bytes) {
  rq_status st = check_cache(c);
  if (st != RQ_OK) return st;
  if (n_tokens < 1 || n_tokens > c->capacity)
    return fail(RQ_EINVAL, "n_tokens %d outside 1..%d", n_tokens, c->capacity);
  if (!bytes) return fail(RQ_EINVAL, "bytes is NULL");
  // the largest over the layers (their kv-heads share the grid by cost)
  uint64_t most = 0;
  for (int l = 0; l < c->n_layers; ++l) {
    const uint64_t b = attn_ws_bytes(c, plan_splits(c, l, n_tokens));
    most = b > most ? b : most;
  }
  *bytes = most;
  return ok();
}

rq_status rq_decode_attention(const rq_cache* c, int32_t layer,
                              int32_t n_tokens, const void* q, float* out,
                              float scale, void* ws, uint64_t ws_bytes,
                              rq_stream stream) {
  rq_status st = check_cache(c);
  if (st != RQ_OK) return st;
  if (!ws) return fail(RQ_EINVAL, "NULL workspace");
  const uint64_t cb = attn_counter_bytes(c);
  if (ws_bytes < cb)
    return fail(RQ_ESMALLWS, "workspace %llu bytes < %llu needed",
                (unsigned long long)ws_bytes, (unsigned long long)cb);
  return rq::decode_attention(c, layer, n_tokens, q, out, scale, ws, cb,
                              reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + cb),
                              ws_bytes - cb, stream);
}

rq_status rq_decode_step(const rq_cache* c, int32_t layer, int32_t n_past, const void* k,
                         const void* v, const void* q, float* out, float scale, void* ws,
                         uint64_t ws_bytes, rq_stream stream) {
  rq_status st = check_cache(c);
  if (st != RQ_OK) return st;
  if (n_past < 0 || n_past >= c->capacity)
    return fail(RQ_EINVAL, "n_past %d outside 0..%d", n_past, c->capacity - 1);
  if (!k || !v) return fail(RQ_EINVAL, "NULL new token");
  if (!ws) return fail(RQ_EINVAL, "NULL workspace");
  const uint64_t cb = rq::decode_counter_bytes(c);
  if (ws_bytes < cb)
    return fail(RQ_ESMALLWS, "workspace of %llu bytes holds no counters (%llu)",
                (unsigned long long)ws_bytes, (unsigned long long)cb);
  float* part = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + cb);
  // everything is checked before the first launch
  st = rq::decode_attention(c, layer, n_past + 1, q, out, scale, ws, cb, part, ws_bytes - cb,
                            stream, k, v, false);
  if (st != RQ_OK) return st;
  // the block that leaves the window (if any) is quantized first; the new
  // token itself goes to the window inside the attention kernel
  const rq::QuantLaunch ql = quant_launch(c, layer, n_past, k, v, 1);
  hipError_t e = rq::launch_quantize(ql, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "quantize launch");
  return rq::decode_attention(c, layer, n_past + 1, q, out, scale, ws, cb, part, ws_bytes - cb,
                              stream, k, v, true);
}

rq_status rq_calibrate_workspace(int32_t n_comp, int32_t n_tokens,
                                 int32_t n_bits, uint64_t* bytes) {
  if (n_comp < 1 || n_tokens < rq::kChunk || n_tokens % rq::kChunk ||
      n_bits < 1 || n_bits > 16 || !bytes)
    return fail(RQ_EINVAL, "bad calibration shape (%d, %d, %d)", n_comp,
                n_tokens, n_bits);
  *bytes = (uint64_t)n_comp * n_bits * sizeof(double) *
           ((uint64_t)n_tokens / rq::kChunk + 1);
  return ok();
}

rq_status rq_calibrate_distortion(int32_t family, int32_t dtype, const void* x,
                                  int32_t n_comp, int32_t n_tokens,
                                  int32_t is_value, const int32_t* bits,
                                  int32_t n_bits, const void* rotation,
                                  const float* codebook, double* mse, double* alpha,
                                  double* beta, double* r2, void* ws,
                                  uint64_t ws_bytes, rq_stream stream) {
  if (family != RQ_KIVI && family != RQ_QUAROT && family != RQ_TURBO &&
      family != RQ_RTN && family != RQ_KIVI_RTN)
    return fail(RQ_EINVAL, "unknown family %d", family);
  // the mixed family sweeps its keys as KIVI and its values as RTN
  if (family == RQ_KIVI_RTN) family = is_value ? RQ_RTN : RQ_KIVI;
  if (family == RQ_TURBO && (!rotation || !codebook))
    return fail(RQ_EINVAL, "TurboQuant needs the rotation and codebook pointers");
  if (dtype != RQ_F16 && dtype != RQ_BF16)
    return fail(RQ_EINVAL, "unknown dtype %d", dtype);
  uint64_t need = 0;
  rq_status st = rq_calibrate_workspace(n_comp, n_tokens, n_bits, &need);
  if (st != RQ_OK) return st;
  if (!x || !bits || !mse || !ws) return fail(RQ_EINVAL, "NULL pointer");
  if ((alpha || beta || r2) && n_bits < 2)
    return fail(RQ_EINVAL, "the fit needs at least two bit-widths");
  const int lo = (family == RQ_QUAROT || family == RQ_RTN) ? 2 : 1;
  for (int j = 0; j < n_bits; ++j) {
    if (bits[j] < lo || bits[j] > 8)
      return fail(RQ_EINVAL, "bit-width %d outside %d..8", bits[j], lo);
    for (int i = 0; i < j; ++i)
      if (bits[i] == bits[j]) return fail(RQ_EINVAL, "repeated bit-width %d", bits[j]);
  }
  if (ws_bytes < need)
    return fail(RQ_ESMALLWS, "workspace %llu bytes < %llu needed",
                (unsigned long long)ws_bytes, (unsigned long long)need);
  rq::CalibLaunch a{};
  a.x = static_cast<const uint16_t*>(x);
  a.mse = static_cast<double*>(ws);
  a.partial = a.mse + (uint64_t)n_comp * n_bits;
  a.n_comp = n_comp;
  a.T = n_tokens;
  a.n_bits = n_bits;
  a.is_value = is_value != 0;
  a.is_bf16 = dtype == RQ_BF16;
  a.family = family;
  a.rot = static_cast<const uint16_t*>(rotation);
  a.cb = codebook;
  for (int j = 0; j < n_bits; ++j) a.bits[j] = (uint8_t)bits[j];
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = rq::launch_calibrate(a, s);
  if (e != hipSuccess) return hip_fail(e, "calibration launch");
  e = hipMemcpyAsync(mse, a.mse, sizeof(double) * n_comp * n_bits,
                     hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return hip_fail(e, "calibration copy");
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "calibration sync");
  if (alpha || beta || r2) {
    std::vector<double> al(n_comp), be(n_comp), rr(n_comp);
    rq::fit_distortion(mse, n_comp, bits, n_bits, al.data(), be.data(), rr.data());
    for (int i = 0; i < n_comp; ++i) {
      bool pos = true;
      for (int j = 0; j < n_bits; ++j) pos = pos && mse[(size_t)i * n_bits + j] > 0;
      if (!pos) al[i] = be[i] = rr[i] = NAN;
      if (alpha) alpha[i] = al[i];
      if (beta) beta[i] = be[i];
      if (r2) r2[i] = rr[i];
    }
  }
  return ok();
}

rq_status rq_turbo_codebook(float* table) {
  if (!table) return fail(RQ_EINVAL, "table is NULL");
  const float* t = rq::turbo_table();
  for (int i = 0; i < RQ_TURBO_TABLE_FLOATS; ++i) table[i] = t[i];
  return ok();
}

rq_status rq_fit_distortion(const double* mse, int32_t n_comp,
                            const int32_t* bits, int32_t n_bits, double* alpha,
                            double* beta, double* r2) {
  if (!mse || !bits || n_comp < 1 || n_bits < 2)
    return fail(RQ_EINVAL, "need mse, bits, n_comp >= 1 and n_bits >= 2");
  bool distinct = false;
  for (int j = 1; j < n_bits; ++j) distinct = distinct || bits[j] != bits[0];
  if (!distinct) return fail(RQ_EINVAL, "bit-widths must not all be equal");
  for (int64_t i = 0; i < (int64_t)n_comp * n_bits; ++i)
    if (!(mse[i] > 0) || !std::isfinite(mse[i]))
      return fail(RQ_EINVAL, "mse[%lld] = %g is not a positive finite number",
                  (long long)i, mse[i]);
  rq::fit_distortion(mse, n_comp, bits, n_bits, alpha, beta, r2);
  return ok();
}

rq_status rq_allocate_bits(int32_t n, const double* w, const double* alpha,
                           const double* beta, double avg_bits, int32_t bmin,
                           int32_t bmax, int32_t* bits_out,
                           double* bits_cont_out, double* J_out) {
  if (n < 1 || !w || !alpha || !beta || !bits_out)
    return fail(RQ_EINVAL, "need n >= 1 and w, alpha, beta, bits_out");
  if (bmin < 1 || bmax > 8 || bmin > bmax)
    return fail(RQ_EINVAL, "bounds [%d, %d] must satisfy 1 <= bmin <= bmax <= 8",
                bmin, bmax);
  if (!std::isfinite(avg_bits)) return fail(RQ_EINVAL, "avg_bits not finite");
  for (int i = 0; i < n; ++i) {
    if (!(w[i] > 0) || !std::isfinite(w[i]) || !(alpha[i] > 0) ||
        !std::isfinite(alpha[i]) || !(beta[i] > 1) || !std::isfinite(beta[i]))
      return fail(RQ_EINVAL, "component %d: need w > 0, alpha > 0, beta > 1", i);
  }
  const int64_t B = rq::budget(n, avg_bits);
  if (B < (int64_t)n * bmin || B > (int64_t)n * bmax)
    return fail(RQ_EINFEASIBLE, "budget %lld outside [%lld, %lld]", (long long)B,
                (long long)n * bmin, (long long)n * bmax);
  rq::greedy(n, w, alpha, beta, B, bmin, bmax, bits_out);
  if (bits_cont_out) rq::waterfill(n, w, alpha, beta, B, bmin, bmax, bits_cont_out);
  if (J_out) {
    double J = 0;
    for (int i = 0; i < n; ++i) J += w[i] * alpha[i] * std::pow(beta[i], -(double)bits_out[i]);
    *J_out = J;
  }
  return ok();
}

rq_status rq_sensitivity_workspace(int32_t gdtype, int32_t n_seq,
                                   int32_t n_comp, int32_t n_tokens,
                                   uint64_t* bytes) {
  if (gdtype != RQ_F32 && gdtype != RQ_F16 && gdtype != RQ_BF16)
    return fail(RQ_EINVAL, "unknown gradient dtype %d", gdtype);
  if (n_seq < 1 || n_seq > 65535 || n_comp < 1 || n_comp > 65535 ||
      n_tokens < 1 || !bytes)
    return fail(RQ_EINVAL, "bad sensitivity shape (%d, %d, %d)", n_seq, n_comp,
                n_tokens);
  const int64_t vecs = (int64_t)n_tokens * rq::kD * (gdtype == RQ_F32 ? 4 : 2) / 16;
  const int64_t chunks = (vecs + rq::kSensChunkVecs - 1) / rq::kSensChunkVecs;
  if (chunks > 0x7fffffff) return fail(RQ_EINVAL, "n_tokens %d too large", n_tokens);
  *bytes = sizeof(double) * ((uint64_t)n_seq * n_comp * chunks + n_comp);
  return ok();
}

rq_status rq_sensitivity(int32_t gdtype, const void* grad, int32_t n_seq,
                         int32_t n_comp, int32_t n_tokens, double* w,
                         void* ws, uint64_t ws_bytes, rq_stream stream) {
  uint64_t need = 0;
  rq_status st = rq_sensitivity_workspace(gdtype, n_seq, n_comp, n_tokens, &need);
  if (st != RQ_OK) return st;
  if (!grad || !w || !ws) return fail(RQ_EINVAL, "NULL pointer");
  if (reinterpret_cast<uintptr_t>(grad) % 16)
    return fail(RQ_EINVAL, "gradient pointer is not 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(ws) % 8)
    return fail(RQ_EINVAL, "workspace pointer is not 8-byte aligned");
  if (ws_bytes < need)
    return fail(RQ_ESMALLWS, "workspace %llu bytes < %llu needed",
                (unsigned long long)ws_bytes, (unsigned long long)need);
  rq::SensLaunch a{};
  a.grad = grad;
  a.slab_vecs = (int64_t)n_tokens * rq::kD * (gdtype == RQ_F32 ? 4 : 2) / 16;
  a.chunks = (int)((a.slab_vecs + rq::kSensChunkVecs - 1) / rq::kSensChunkVecs);
  a.w = static_cast<double*>(ws);
  a.partial = a.w + n_comp;
  a.n_seq = n_seq;
  a.n_comp = n_comp;
  a.T = n_tokens;
  a.dtype = gdtype;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = rq::launch_sensitivity(a, s);
  if (e != hipSuccess) return hip_fail(e, "sensitivity launch");
  e = hipMemcpyAsync(w, a.w, sizeof(double) * n_comp, hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return hip_fail(e, "sensitivity copy");
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "sensitivity sync");
  return ok();
}

rq_status rq_cap_weights(int32_t n, double* w, double factor) {
  if (n < 1 || !w) return fail(RQ_EINVAL, "need n >= 1 weights");
  if (!std::isfinite(factor) || !(factor > 0))
    return fail(RQ_EINVAL, "cap factor must be finite and > 0");
  double sum = 0.0;
  for (int i = 0; i < n; ++i) {
    if (!std::isfinite(w[i]) || w[i] < 0)
      return fail(RQ_EINVAL, "weight %d is not finite and >= 0", i);
    sum += w[i];
  }
  const double cap = factor * (sum / n);
  for (int i = 0; i < n; ++i) w[i] = w[i] < cap ? w[i] : cap;
  return ok();
}

rq_status rq_fallback_beta(int32_t n, double* beta, const double* r2,
                           double r2_min) {
  if (n < 1 || !beta || !r2) return fail(RQ_EINVAL, "need n >= 1 components");
  if (!std::isfinite(r2_min)) return fail(RQ_EINVAL, "r2_min is not finite");
  double sum = 0.0;
  for (int i = 0; i < n; ++i) {
    if (!std::isfinite(beta[i]) || !std::isfinite(r2[i]))
      return fail(RQ_EINVAL, "component %d: beta or r2 is not finite", i);
    sum += beta[i];
  }
  const double mean = sum / n;
  for (int i = 0; i < n; ++i)
    if (r2[i] < r2_min && mean < beta[i]) beta[i] = mean;
  return ok();
}

}  // extern "C"
