// Decode attention without a caller workspace: the arrival counters and
// partial results live in a file-scope device array of the library, one
// copy per GPU, so the call allocates nothing (for callers that cannot
// allocate device memory, e.g. under stream capture or in serving loops).
#include <mutex>

#include "rq_internal.h"

namespace rq {
namespace {

// Counters first (zero at load; each call tags them with its number), then
// the partials.
constexpr uint64_t kScratchCounterBytes = 1ull << 20;
constexpr uint64_t kScratchBytes = 8ull << 20;
static_assert(kScratchCounterBytes % 256 == 0, "partials stay 256-byte aligned");

__device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices];

// This device's copy of the scratch array (looked up once per device, with
// the device current).
rq_status scratch_ptr(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return set_error(RQ_EDEVICE, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices) return set_error(RQ_EUNSUPPORTED, "device index above 63");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return set_error(RQ_EDEVICE, "hipGetSymbolAddress of the attention scratch failed");
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return RQ_OK;
}

}  // namespace
}  // namespace rq

extern "C" {

uint64_t rq_decode_static_bytes(void) { return rq::kScratchBytes; }

rq_status rq_decode_attention_static(const rq_cache* c, int32_t layer, int32_t n_tokens,
                                     const void* q, float* out, float scale,
                                     rq_stream stream) {
  void* p = nullptr;
  const rq_status st = rq::scratch_ptr(&p);
  if (st != RQ_OK) return st;
  uint8_t* base = static_cast<uint8_t*>(p);
  return rq::decode_attention(c, layer, n_tokens, q, out, scale,
                              base, rq::kScratchCounterBytes,
                              reinterpret_cast<float*>(base + rq::kScratchCounterBytes),
                              rq::kScratchBytes - rq::kScratchCounterBytes, stream);
}

}  // extern "C"
