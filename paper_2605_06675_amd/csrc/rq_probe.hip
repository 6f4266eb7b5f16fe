// Streaming-read probe: the HBM read rate a plain kernel reaches on this
// device, the ceiling the path's kernels are measured against.  Each thread
// reads 16-byte vectors with non-temporal loads (eight in flight), folds
// them with XOR and writes one word per workgroup, so the bytes read are
// the only traffic that matters.
#include "rq_device.h"
#include "rq_internal.h"

namespace rq {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 8;

__global__ void __launch_bounds__(kProbeThreads)
read_probe_kernel(const u4* src, uint64_t n_vec, uint32_t* sink) {
  const RQ_GLOBAL u4* p = gptr(src);
  const uint64_t stride = (uint64_t)gridDim.x * kProbeThreads * kProbeUnroll;
  uint32_t x = 0;
  for (uint64_t base = (uint64_t)blockIdx.x * kProbeThreads * kProbeUnroll + threadIdx.x;
       base < n_vec; base += stride) {
    u4 v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) {
      const uint64_t i = base + (uint64_t)u * kProbeThreads;
      v[u] = i < n_vec ? __builtin_nontemporal_load(p + i) : (u4){0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (int d = 32; d >= 1; d >>= 1) x ^= __shfl_xor(x, d, 64);
  __shared__ uint32_t ws[kProbeThreads / 64];
  if ((threadIdx.x & 63) == 0) ws[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = ws[0] ^ ws[1] ^ ws[2] ^ ws[3];
}

}  // namespace
}  // namespace rq

extern "C" rq_status rq_read_probe(const void* buf, uint64_t bytes, uint32_t* sink,
                                   int32_t n_blocks, rq_stream stream) {
  if (!buf || !sink || bytes < 16 || bytes % 16 || n_blocks < 1 || n_blocks > 65535)
    return rq::set_error(RQ_EINVAL, "read probe: need a 16-byte multiple, a sink and 1..65535 blocks");
  if (reinterpret_cast<uintptr_t>(buf) % 16)
    return rq::set_error(RQ_EINVAL, "read probe: buffer not 16-byte aligned");
  hipLaunchKernelGGL(rq::read_probe_kernel, dim3(n_blocks), dim3(rq::kProbeThreads), 0,
                     reinterpret_cast<hipStream_t>(stream), static_cast<const rq::u4*>(buf),
                     bytes / 16, sink);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? RQ_OK : rq::set_error(RQ_EDEVICE, "read probe launch failed");
}
