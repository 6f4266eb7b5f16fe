// Internal declarations shared by the host library and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/rq.h"

namespace rq {

constexpr int kD = 128;          // head_dim
constexpr int kChunk = 32;       // codes per packed chunk = tokens per block
constexpr int kMetaBlockKivi = 512;   // bytes of KIVI metadata per block
constexpr int kMetaBlockTok = 64;     // bytes of per-token metadata per block

// Metadata bytes of one block of kind (0 = K, 1 = V) in a family.
__host__ __device__ constexpr int meta_block_bytes(int family, int kind) {
  return (family == RQ_KIVI || (family == RQ_KIVI_RTN && kind == 0)) ? kMetaBlockKivi
                                                                     : kMetaBlockTok;
}
// Byte offset, inside one layer's metadata, of block 0 of unit (h, kind, b):
// [h][kind][batch][block], a K block taking meta_block_bytes(family, 0)
// bytes and a V block meta_block_bytes(family, 1).
__host__ __device__ inline size_t meta_unit_offset(int family, int h, int kind, int b, int B,
                                                   int nblk_cap) {
  const size_t mk = meta_block_bytes(family, 0), mv = meta_block_bytes(family, 1);
  return (size_t)h * B * nblk_cap * (mk + mv) + (size_t)kind * B * nblk_cap * mk +
         (size_t)b * nblk_cap * (kind ? mv : mk);
}
constexpr int kAttnGroup = 16;        // streaming slots per merge group
constexpr int kAttnMergeFlat = 16;    // at most this many: one merge level
constexpr int kAttnResChunk = 32;     // window tokens per window workgroup
constexpr int kAttnMaxDepth = 4;      // most blocks in flight per attention wave
constexpr int kAttnWaves = 4;         // waves per attention workgroup

// Per-layer view of the bit table: byte offsets of each (head, kind) code
// region and its bit-width.  Passed by value as a kernel argument, so a
// kernel finds its head's width and region in O(1).
struct LayerTable {
  uint64_t code_off[RQ_MAX_KV_HEADS][2];
  uint8_t bits[RQ_MAX_KV_HEADS][2];
};

// Field positions of the packed codes of every width (1..8) in the fp16
// operands the attention kernel builds: key pair slot i (0..15) and value
// slot i (0..3).  Filled by the attention launchers.
struct FieldPosTab {
  int8_t k[9][16];
  int8_t v[9][4];
};

struct RingLaunch {
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* resid;        // this layer's rings
  int B, H, n_new, n_past, R;
  int t_lo, t_hi;         // tokens [t_lo, t_hi) go to the window
};

struct QuantLaunch {
  const uint16_t* k;      // [B][H][n_new][128]
  const uint16_t* v;
  uint8_t* codes;
  uint8_t* meta;          // start of this layer's metadata
  uint16_t* resid;        // start of this layer's residual rings
  int B, H, n_new, n_past, cap, R;
  int blk0, nblk;         // blocks [blk0, blk0 + nblk) get quantized
  int kind_lo, kind_n;    // kinds kind_lo .. kind_lo + kind_n - 1 (K = 0, V = 1)
  RingLaunch ring;        // window rows this launch also copies
  int ring_fused;         // (when set; else the window has its own launch)
  int is_bf16;
  int family;
  int n_cu;               // compute units of the device (grid sizing)
  const uint16_t* rot;    // TurboQuant: this layer's rotations [H][128][128] bf16
  const float* cb;        // TurboQuant: codebook table (rq_turbo_codebook)
  LayerTable tab;
};

struct AttnLaunch {
  const uint16_t* q;      // [B][Hq][128]
  const uint8_t* codes;
  const uint8_t* meta;    // this layer
  const uint16_t* resid;  // this layer
  float* out;             // [B][Hq][128]
  // the token this call appends (fused decode step; t_new < 0: none):
  // [B][H][128] rows of K and V, read for the attention and written to
  // window slot t_new mod (R + 32) of this layer's residual window
  const uint16_t* k_new;
  const uint16_t* v_new;
  uint16_t* resid_w;      // this layer's window, writable
  int t_new;
  float* part;            // [B][H][pstride][G][2 + 128] (max, sum, acc);
                          // slots 0..n_wg-1 streaming, n_wg..n_wg+n_rw-1
                          // the residual window, then one per merge group
  uint64_t* counters;     // [B][H][cstride] arrival and claim counters:
                          // (epoch << 32) | count
  uint32_t epoch;         // this call's number on the workspace (>= 1)
  int pstride;            // partial slots per unit
  int cstride;            // counters per unit: tickets (final, one per
                          // merge group) in the first 128-byte lines, then
                          // one 128-byte line per claim group
  int claim_off;          // first claim counter of a unit (in counters)
  int B, H, G, cap, R;
  int GP;                 // smallest power of two >= G
  int nq, n_tokens;
  int n_wg;               // grid slots per unit: the largest nwg[h]
  uint16_t nwg[RQ_MAX_KV_HEADS];  // workgroups streaming blocks, per kv-head
  int n_rw;               // workgroups per unit on the 16-bit window
  int wave_bytes;         // LDS bytes of one wave's block ring
  int area_bytes;         // LDS bytes of the ring/merge/staging area
  int is_bf16, family;
  float qscale;           // scale * log2(e)
  const uint16_t* rot;    // TurboQuant: this layer's rotations [H][128][128] bf16
  const float* cb;        // TurboQuant: codebook table (rq_turbo_codebook)
  LayerTable tab;
  FieldPosTab fpos;
};

struct CalibLaunch {
  const uint16_t* x;      // [n_comp][T][128]
  double* partial;        // [n_comp][n_blk][n_bits]
  double* mse;            // [n_comp][n_bits]
  int n_comp, T, n_bits, is_value, is_bf16, family;
  uint8_t bits[16];
  const uint16_t* rot;    // TurboQuant: [n_comp][128][128] bf16
  const float* cb;        // TurboQuant: codebook table
};

hipError_t launch_quantize(const QuantLaunch& a, hipStream_t s);
hipError_t launch_quantize_turbo(const QuantLaunch& a, hipStream_t s);
hipError_t launch_ring(const RingLaunch& a, hipStream_t s);
hipError_t launch_attention(const AttnLaunch& a, hipStream_t s);
// LDS of the attention kernel: the area (the waves' block rings while
// streaming; the wave merge, window staging and merging scratch after or
// instead), then the 16-bit query rows and, for TurboQuant, the rotated
// query rows.  attention_area_bytes: the area for rings of wave_bytes each.
size_t attention_area_bytes(int G, int wave_bytes, int family);
size_t attention_lds_bytes(int G, int wave_bytes, int family);
// LDS after the area: G 16-bit query rows, then (TurboQuant) G rotated rows
size_t attention_tail_bytes(int G, int family);
hipError_t launch_calibrate(const CalibLaunch& a, hipStream_t s);

constexpr int kSensChunkVecs = 8192;  // 16-byte vectors per sensitivity workgroup

struct SensLaunch {
  const void* grad;       // [n_seq][n_comp][T][128] in dtype
  double* partial;        // [n_seq][n_comp][chunks]
  double* w;              // [n_comp]
  int64_t slab_vecs;      // 16-byte vectors per (sequence, component)
  int n_seq, n_comp, T, chunks, dtype;
};
hipError_t launch_sensitivity(const SensLaunch& a, hipStream_t s);

// Decode attention of one layer with the arrival counters (counter_cap
// bytes, epoch-tagged) and the partial results (part_cap bytes) in the
// given device buffers: the validation and launch shared by the entry
// points with a caller's workspace and with the library's own scratch.
// k_new, v_new: the token this call appends at position n_tokens - 1 (a
// fused decode step whose flush, if any, has been launched), or NULL.
// launch = false: validate only.
rq_status decode_attention(const rq_cache* c, int32_t layer, int32_t n_tokens, const void* q,
                           float* out, float scale, void* counters, uint64_t counter_cap,
                           float* part, uint64_t part_cap, rq_stream stream,
                           const void* k_new = nullptr, const void* v_new = nullptr,
                           bool launch = true);
// Bytes of arrival counters a cache's calls use.
uint64_t decode_counter_bytes(const rq_cache* c);
// Record an error message for rq_last_error and return code.
rq_status set_error(rq_status code, const char* msg);

}  // namespace rq
