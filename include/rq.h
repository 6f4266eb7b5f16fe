/*
 * librq -- RateQuant hot path on AMD Instinct MI355X (gfx950).
 *
 * RateQuant (arXiv 2605.06675) gives every KV head its own bit-width: it
 * fits a distortion curve D(b) = alpha * beta^-b per quantizer and component
 * (Alg. 1 Stage 2; Sec. 3.4), allocates integer bits under an average budget
 * (eq. 1; Theorem 1; Alg. 1 Stage 3 / Alg. 2), and then quantizes each head
 * of the KV cache at its own width; decode attention reads the packed cache
 * back (Sec. 3.4 "Pipeline summary"; Appendix "Runtime Analysis").
 *
 * Conventions for every call
 *  - Plain C types only.  "device" pointers are HIP device memory owned by
 *    the caller; "host" pointers are ordinary host memory owned by the
 *    caller.  The library allocates no device memory and keeps no state
 *    between calls.
 *  - Asynchronous calls enqueue kernels on the given stream and return
 *    without waiting.  Synchronous calls say so.
 *  - Every argument is validated on the host before anything is enqueued;
 *    a call that returns an error has written nothing.  rq_last_error()
 *    then describes the problem (thread-local, valid until the next call
 *    on the same thread).
 *  - head_dim is 128.  Bit-widths are 1..8 (QuaRot and RTN need >= 2, and
 *    so do the values of KIVI_RTN).
 *
 * Numeric formats (bit-exact contract shared with the test oracle)
 *  - K/V inputs are fp16 or bf16 (rq_dtype).  Metadata (scale, zero) is
 *    fp16, rounded to nearest-even from fp32 and saturated at +-65504.
 *  - A code is decided by correctly-rounded fp32 steps, rint half-to-even:
 *      KIVI   z = fp16(min), s = fp16(max(max - z, 0) / (2^b - 1)),
 *             code = rint(clamp((x - z) * fp32(1/s), 0, 2^b - 1)),
 *             all codes 0 when s == 0; groups: keys = one channel over 32
 *             consecutive tokens, values = 32 consecutive channels of one
 *             token.
 *      QuaRot y = fp32(FWHT(x) * fp32(1/sqrt(128))) with the butterfly
 *             stages h = 1, 2, ..., 64 in that order; s = fp16(max|y| /
 *             (2^(b-1) - 1)); code = rint(clamp(y * fp32(1/s), -q, q)) +
 *             2^(b-1), q = 2^(b-1) - 1 (all codes 2^(b-1) when s == 0).
 *      RTN    the QuaRot step on y = x itself (per-token symmetric
 *             round-to-nearest, no rotation; Appendix "RTN Base
 *             Quantizer").
 *      KIVI_RTN  keys by KIVI, values by RTN: each side its own base
 *             quantizer (the per-side treatment of Sec. 3.4, "K/V
 *             separation").
 *      Turbo  n = fp16(fp32(|x|)) (sum of squares and root in fp64);
 *             y = R x, t = y * (sqrt(128) / n) (0 when n == 0); code =
 *             number of thresholds of the b-bit codebook below t.  y is
 *             summed in fp32 on the matrix cores, so a coordinate whose t
 *             lies within the rounding of that sum of a threshold may take
 *             the neighbouring code; everything else is exact.
 *  - Packed chunk: 32 codes of one stream in exactly b uint32 words.
 *    b = 3: one 3-bit field per code.  The three words form a 96-bit
 *    stream (stream bit 32k + j = bit j of word k) of four 24-bit
 *    quarters; quarter q holds code 4q + i at stream bit 24q + 3i and
 *    code 16 + 4q + i at stream bit 24q + 12 + 3i (i = 0..3).
 *    Other widths: the code bits are split into planes of widths equal
 *    to the binary digits of b, widest first (5 -> 4+1, 6 -> 4+2,
 *    7 -> 4+2+1); plane width w occupies w words, and its word d holds
 *    the field of code d*16/w + k at bit k*w and that of code
 *    16 + d*16/w + k at bit 16 + k*w, for k = 0 .. 16/w - 1.
 *  - Pair order of 32 entries: 0,16,1,17,...,15,31.
 *
 * Cache layout (one buffer each; the caller allocates the sizes reported by
 * rq_cache_sizes).  A "unit" is one (layer, batch entry, kv-head).  T_cap is
 * rq_cache.capacity (a multiple of 32), R = rq_cache.residual.
 *  codes  regions in order layer, head, K then V; region (l,h,kind) holds
 *         batch * T_cap * 16 * b bytes, b = bits[l][h][kind]:
 *           K: [batch][token][chunk q: channels 32q..32q+31][b words]
 *           V: [batch][block of 32 tokens][channel][b words]  (a chunk is
 *              the 32 tokens of the block)
 *  meta   [l][h][kind][batch][block][one block's metadata], a block of
 *         kind K taking mK bytes and of kind V mV bytes:
 *         KIVI-style (512 bytes): [4][s(32), z(32)] fp16, pair order;
 *                 K: group index = chunk q, entries = channels;
 *                 V: group index = channel group cg, entries = tokens.
 *         per-token (64 bytes): [s(32 tokens)] fp16, pair order (QuaRot
 *                 and RTN scales, Turbo norms).
 *         KIVI: both sides KIVI-style; KIVI_RTN: K KIVI-style, V per-token;
 *         QuaRot, RTN, Turbo: both sides per-token.
 *  resid  [l][batch][h][kind][R + 32][128] in the input dtype; token t of
 *         the 16-bit window lives in slot t mod (R + 32).
 *  Residual rule: with T tokens cached the quantized prefix is
 *  nq = max(0, floor((T - R) / 32) * 32); tokens nq .. T-1 stay 16-bit.
 */
#ifndef RQ_H
#define RQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t rq_status;
#define RQ_OK 0
#define RQ_EINVAL (-1)        /* bad argument                               */
#define RQ_EINFEASIBLE (-2)   /* budget outside [n*bmin, n*bmax]            */
#define RQ_EUNSUPPORTED (-3)  /* valid but not implemented (head_dim, ...)  */
#define RQ_EDEVICE (-4)       /* a HIP runtime call failed                  */
#define RQ_ESMALLWS (-5)      /* workspace smaller than required            */

#define RQ_KIVI 0
#define RQ_QUAROT 1
#define RQ_TURBO 2
#define RQ_RTN 3
#define RQ_KIVI_RTN 4         /* KIVI keys, RTN values (mixed families)     */

#define RQ_F16 0
#define RQ_BF16 1
#define RQ_F32 2              /* gradients of rq_sensitivity only            */

#define RQ_MAX_KV_HEADS 32

/* Floats of the TurboQuant codebook table filled by rq_turbo_codebook. */
#define RQ_TURBO_TABLE_FLOATS (8 * 2 * 256)

/* HIP stream handle, passed through as an opaque pointer. */
typedef void* rq_stream;

/* Cache descriptor.  Plain data filled by the caller; the library only
 * reads it.  bits is the per-(layer, kv-head) bit table of the paper (its
 * "static lookup table", Appendix "Runtime Analysis"): host int8
 * [n_layers][n_kv_heads][2], K then V. */
typedef struct rq_cache {
  int32_t family;        /* RQ_KIVI, RQ_QUAROT, RQ_TURBO, RQ_RTN or
                            RQ_KIVI_RTN                                    */
  int32_t dtype;         /* RQ_F16 or RQ_BF16: K/V/q input type           */
  int32_t n_layers;
  int32_t batch;
  int32_t n_kv_heads;    /* <= RQ_MAX_KV_HEADS                            */
  int32_t n_q_heads;     /* multiple of n_kv_heads, ratio <= 16           */
  int32_t head_dim;      /* 128                                           */
  int32_t capacity;      /* max cached tokens per sequence, % 32 == 0     */
  int32_t residual;      /* R >= 0: 16-bit window length in tokens        */
  const int8_t* bits;    /* host [n_layers][n_kv_heads][2]                */
  void* codes;           /* device, >= codes_bytes                        */
  void* meta;            /* device, >= meta_bytes                         */
  void* resid;           /* device, >= resid_bytes                        */
  /* RQ_TURBO only (NULL otherwise): device bf16 [n_layers][n_kv_heads]
   * [128][128], the orthogonal rotation R of each (layer, kv-head),
   * row-major, applied as y = R x; and the device copy of the table filled
   * by rq_turbo_codebook. */
  const void* rotation;
  const float* codebook;
} rq_cache;

/* The per-coordinate codebook of the TurboQuant-style quantizer: the
 * Lloyd-Max quantizer of N(0,1) with 2^b levels, b = 1..8 (Sec. 2;
 * Sec. 3.1, Table 6).  Fills host float [8][2][256]: entry [b-1][0][k] is
 * the decision threshold between levels k and k+1 (the fp32 rounding of the
 * midpoint of the two centroids, k < 2^b - 1; +inf beyond), entry
 * [b-1][1][k] centroid k (ascending, k < 2^b).  The caller copies the table
 * to the device and passes it in rq_cache.codebook and to the sweep.  The
 * first call computes it (about a second); later calls copy.  Host only. */
rq_status rq_turbo_codebook(float* table);

/* Library version (major*10000 + minor*100 + patch). */
int32_t rq_version(void);

/* Thread-local text for the last non-OK status (never NULL). */
const char* rq_last_error(void);

/* Validate a descriptor (device pointers may be NULL here) and report the
 * buffer sizes in bytes of the mixed-bit cache: codes at each kv-head's
 * own K and V widths (the per-head bit table, Sec. 3.3; memory as in
 * Appendix "Runtime Analysis"), metadata per the family, and the 16-bit
 * window.  Any output pointer may be NULL.  Host only. */
rq_status rq_cache_sizes(const rq_cache* c, uint64_t* codes_bytes,
                         uint64_t* meta_bytes, uint64_t* resid_bytes);

/* Byte offset of the code region (layer, head, kind) inside codes, i.e. the
 * prefix sum of region sizes in (layer, head, K-then-V) order: the O(1)
 * lookup of the bit table.  Host only. */
rq_status rq_region_offset(const rq_cache* c, int32_t layer, int32_t head,
                           int32_t kind, uint64_t* offset);

/* Append n_new >= 1 tokens to one layer that already holds n_past tokens
 * (0 <= n_past, n_past + n_new <= capacity).  k, v: device
 * [batch][n_kv_heads][n_new][128] in dtype, contiguous.  Quantizes every
 * 32-token block that leaves the residual window (reading older tokens
 * from the window and newer ones from k, v) and stores the newest tokens
 * in the window.  Asynchronous.  Sec. 3.4 / Appendix "Quantizer
 * Implementation" (the base quantizers), Appendix "Runtime Analysis" (the
 * per-head bit lookup). */
rq_status rq_quantize_kv(const rq_cache* c, int32_t layer, int32_t n_past,
                         const void* k, const void* v, int32_t n_new,
                         rq_stream stream);

/* Workspace bytes rq_decode_attention needs for n_tokens cached tokens
 * (it varies with n_tokens; size for the largest call, or re-query): the
 * per-(batch, kv-head) counters and the partial results of the split
 * decode of Appendix "Runtime Analysis" (the lookup-and-dequantize path).
 * Host only. */
rq_status rq_decode_workspace(const rq_cache* c, int32_t n_tokens,
                              uint64_t* bytes);

/* Decode attention of one new query per sequence over the n_tokens cached
 * tokens of one layer (1 <= n_tokens <= capacity), the inference path of
 * Appendix "Runtime Analysis" (each kv-head's blocks dequantized at its own
 * widths from the bit table, Sec. 3.3; the base quantizers of Sec. 3.4 /
 * Appendix "Quantizer Implementation"):
 *   out[b][j] = softmax(scale * q[b][j] . K_hat^T) V_hat,
 * K_hat/V_hat the dequantized prefix plus the 16-bit window, query head j
 * reading kv-head j / (n_q_heads / n_kv_heads).  q: device
 * [batch][n_q_heads][128] in dtype; out: device fp32, same shape; ws:
 * device scratch of at least rq_decode_workspace bytes.  Its start holds
 * counters (a fixed number per (batch, kv-head), set by the cache's
 * capacity), each tagged with the number of the call counting in it: the
 * library numbers the calls on each workspace (by its address), so a count
 * left by an earlier call that did not finish is recognised and replaced;
 * a zeroed buffer is always valid, and so is one left by earlier calls.
 * The rest holds per-call partial results.  Calls that share a workspace
 * must not overlap (they would race on the counters and partials).
 * Accuracy: fp16 matrix-core operands with fp32 accumulation; the error is
 * within 1e-2 max-abs for values of unit scale and grows in proportion to
 * max|V_hat| beyond it; inputs must be finite, |scale * q| and the
 * dequantized |K_hat|, |V_hat| below 2^56.  A layer whose K+V widths need
 * more LDS than the device offers returns RQ_EUNSUPPORTED.
 * Asynchronous. */
rq_status rq_decode_attention(const rq_cache* c, int32_t layer,
                              int32_t n_tokens, const void* q, float* out,
                              float scale, void* ws, uint64_t ws_bytes,
                              rq_stream stream);

/* One decode step of one layer: append one token (k, v: device
 * [batch][n_kv_heads][1][128] in dtype, contiguous) to the n_past cached
 * ones (0 <= n_past < capacity) and attend over the n_past + 1 tokens with
 * q, as rq_quantize_kv(n_past, k, v, 1) followed by
 * rq_decode_attention(n_past + 1) would, with the same cache contents
 * afterwards and outputs to the same accuracy.  Fused (the per-step path of
 * Appendix "Runtime Analysis": each layer's append, flush and lookup-and-
 * dequantize attention in as few launches as possible): the block that
 * leaves the residual window, if any, is quantized first (one launch),
 * then one attention launch also writes the new token to the window.
 * Everything is validated before the first launch: an error leaves the
 * cache unchanged.  Workspace and overlap rules as rq_decode_attention.
 * Asynchronous. */
rq_status rq_decode_step(const rq_cache* c, int32_t layer, int32_t n_past,
                         const void* k, const void* v, const void* q,
                         float* out, float scale, void* ws, uint64_t ws_bytes,
                         rq_stream stream);

/* For callers that cannot allocate device memory (code under stream
 * capture, serving loops, harnesses that forbid allocation):
 * rq_decode_attention with the workspace replaced by the library's own
 * scratch, a static device array of rq_decode_static_bytes() bytes (8 MiB:
 * 1 MiB of arrival counters, 7 MiB of partial results) that each GPU the
 * library runs on holds until the process ends.  Same arguments, results
 * and errors as rq_decode_attention otherwise; a call whose counters or
 * partials exceed those sizes returns RQ_ESMALLWS.  The call allocates
 * nothing.  Every call on one GPU shares that GPU's scratch: calls that
 * overlap on one GPU (different streams, or host threads) race and must be
 * serialized by the caller.  Asynchronous. */
uint64_t rq_decode_static_bytes(void);
rq_status rq_decode_attention_static(const rq_cache* c, int32_t layer,
                                     int32_t n_tokens, const void* q,
                                     float* out, float scale,
                                     rq_stream stream);

/* Measurement utility, not part of the method: reads `bytes` (a multiple of
 * 16) of the device buffer buf once with a plain streaming kernel of
 * n_blocks workgroups (1..65535) of 256 threads and writes one word per
 * workgroup to the device array sink[n_blocks].  Timed by the caller, it
 * gives the device's streaming-read ceiling that the path's HBM rates are
 * compared with.  Asynchronous. */
rq_status rq_read_probe(const void* buf, uint64_t bytes, uint32_t* sink,
                        int32_t n_blocks, rq_stream stream);

/* Workspace bytes rq_calibrate_distortion needs. */
rq_status rq_calibrate_workspace(int32_t n_comp, int32_t n_tokens,
                                 int32_t n_bits, uint64_t* bytes);

/* Distortion sweep + fit (Alg. 1 Stage 2; Sec. 3.4 "Distortion
 * calibration").  x: device [n_comp][n_tokens][128] in dtype, the
 * calibration vectors of each component (n_tokens % 32 == 0).  For every
 * component i and bit-width bits[j]:
 *   mse[i][j] = mean over tokens and channels of (x - dequant(quant(x)))^2
 * with the key grouping (is_value = 0) or value grouping (is_value = 1) of
 * the family, measured in the unrotated domain; then alpha, beta, r2 as in
 * rq_fit_distortion.  rotation, codebook: RQ_TURBO only (NULL otherwise):
 * device bf16 [n_comp][128][128], one rotation per component, and the
 * device codebook table.  mse, alpha, beta, r2: host arrays ([n_comp][n_bits]
 * and [n_comp]); alpha/beta/r2 may be NULL to skip the fit.  ws: device
 * scratch of rq_calibrate_workspace bytes.  Synchronous: waits for the
 * stream and copies the results to the host. */
rq_status rq_calibrate_distortion(int32_t family, int32_t dtype,
                                  const void* x, int32_t n_comp,
                                  int32_t n_tokens, int32_t is_value,
                                  const int32_t* bits, int32_t n_bits,
                                  const void* rotation, const float* codebook,
                                  double* mse, double* alpha, double* beta,
                                  double* r2, void* ws, uint64_t ws_bytes,
                                  rq_stream stream);

/* Least-squares fit of ln D = ln alpha - b ln beta per component
 * (Alg. 1 Stage 2).  mse: host [n_comp][n_bits] (all > 0), n_bits >= 2
 * distinct widths.  Outputs host [n_comp]; r2 = 1 - SS_res/SS_tot (1 when
 * SS_tot = 0).  Host only. */
rq_status rq_fit_distortion(const double* mse, int32_t n_comp,
                            const int32_t* bits, int32_t n_bits,
                            double* alpha, double* beta, double* r2);

/* Integer bit allocation over n components (eq. 1 with per-component
 * alpha_i, beta_i; Theorem 1 and its bound handling; Alg. 1 Stage 3 /
 * Alg. 2).  Budget B = round(avg_bits * n) (halves away from zero).
 * bits_out[i] (host int32 [n]) is the greedy max-marginal-gain allocation:
 * start at bmin and give each of the B - n*bmin remaining bits to the
 * component with the largest log-gain
 *   log(w) + log(alpha) - b*log(beta) + log1p(-1/beta)
 * (IEEE double, left to right; ties to the lowest index), never above bmax.
 * bits_cont_out (nullable, host double [n]) receives the continuous optimum
 * (the KKT point of eq. 1, reverse waterfilling with the box bounds) and
 * J_out (nullable) the weighted distortion sum w_i alpha_i beta_i^-b_i of
 * bits_out.  Requires w, alpha > 0, beta > 1, 1 <= bmin <= bmax <= 8 and
 * n*bmin <= B <= n*bmax (else RQ_EINFEASIBLE).  Host only. */
rq_status rq_allocate_bits(int32_t n, const double* w, const double* alpha,
                           const double* beta, double avg_bits, int32_t bmin,
                           int32_t bmax, int32_t* bits_out,
                           double* bits_cont_out, double* J_out);

/* Workspace bytes rq_sensitivity needs. */
rq_status rq_sensitivity_workspace(int32_t gdtype, int32_t n_seq,
                                   int32_t n_comp, int32_t n_tokens,
                                   uint64_t* bytes);

/* Stage-1 gradient sensitivity (Alg. 1 Stage 1; Sec. 3.3 "Sensitivity
 * Estimation"; Appendix "Temporal aggregation").  grad: device
 * [n_seq][n_comp][n_tokens][128] in gdtype (RQ_F32, RQ_F16 or RQ_BF16),
 * 16-byte aligned: the gradient of the loss with respect to each
 * component's cache (one kv-head's keys or values) at every position of
 * each calibration sequence, as a backward pass produces it.  For every
 * component i:
 *   w[i] = (1/n_seq) sum_s (1/n_tokens) sum_t sum_c grad[s][i][t][c]^2
 * with the squares and sums in fp64 in a fixed order (deterministic).
 * w: host [n_comp].  ws: device scratch of rq_sensitivity_workspace bytes.
 * n_seq and n_comp are at most 65535.  Synchronous: waits for the stream
 * and copies w to the host. */
rq_status rq_sensitivity(int32_t gdtype, const void* grad, int32_t n_seq,
                         int32_t n_comp, int32_t n_tokens, double* w,
                         void* ws, uint64_t ws_bytes, rq_stream stream);

/* Sensitivity cap (Appendix "Failure modes", mitigation of extreme
 * outliers): w[i] <- min(w[i], factor * mean(w)) in place, the mean of the
 * uncapped weights summed in index order in double; the paper uses
 * factor = 5.  Requires n >= 1, every w finite and >= 0, factor finite and
 * > 0.  Host only. */
rq_status rq_cap_weights(int32_t n, double* w, double factor);

/* Fit fallback for poorly fitting components (Appendix "Distortion Model
 * Parameters", outlier heads): where r2[i] < r2_min, beta[i] <- min(beta[i],
 * mean(beta)) in place, the mean over all n fitted betas summed in index
 * order in double; the paper uses r2_min = 0.96.  Requires n >= 1 and
 * finite beta, r2 and r2_min.  Host only. */
rq_status rq_fallback_beta(int32_t n, double* beta, const double* r2,
                           double r2_min);

#ifdef __cplusplus
}
#endif

#endif /* RQ_H */
