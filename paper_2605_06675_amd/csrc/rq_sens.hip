// Stage-1 sensitivity: the mean over calibration sequences and positions of
// each component's squared gradient norm (Alg. 1 Stage 1; Sec. 3.3
// "Sensitivity Estimation"; Appendix "Temporal aggregation").
//
// A pure HBM stream: every gradient element is read once.  A workgroup owns
// one chunk of one (sequence, component) slab of T x 128 elements, reads it
// with 16-byte loads (eight in flight per thread), squares and sums in fp64
// (the square of an fp32 or 16-bit value is exact in fp64), and writes one
// partial.  A second kernel adds each component's partials in a fixed order,
// so the result does not depend on scheduling.
#include "rq_device.h"
#include "rq_internal.h"

namespace rq {

namespace {

constexpr int kSensThreads = 256;
constexpr int kUnroll = 8;

__device__ __forceinline__ double sq16(uint32_t w, int is_bf16) {
  const double a = (double)widen(w & 0xffffu, is_bf16);
  const double b = (double)widen(w >> 16, is_bf16);
  return __builtin_fma(a, a, b * b);
}

__device__ __forceinline__ double sq_vec(u4 v, int dtype) {
  if (dtype == RQ_F32) {
    const double x0 = (double)__uint_as_float(v.x), x1 = (double)__uint_as_float(v.y);
    const double x2 = (double)__uint_as_float(v.z), x3 = (double)__uint_as_float(v.w);
    return __builtin_fma(x0, x0, x1 * x1) + __builtin_fma(x2, x2, x3 * x3);
  }
  const int bf = dtype == RQ_BF16;
  return (sq16(v.x, bf) + sq16(v.y, bf)) + (sq16(v.z, bf) + sq16(v.w, bf));
}

__global__ void __launch_bounds__(kSensThreads)
sens_kernel(SensLaunch a) {
  const int chunk = blockIdx.x, comp = blockIdx.y, seq = blockIdx.z;
  const size_t slab = (size_t)seq * a.n_comp + comp;
  const RQ_GLOBAL u4* src = gptr(reinterpret_cast<const u4*>(a.grad)) +
                            slab * a.slab_vecs + (size_t)chunk * kSensChunkVecs;
  const int64_t left = a.slab_vecs - (int64_t)chunk * kSensChunkVecs;
  const int nv = left < kSensChunkVecs ? (int)left : kSensChunkVecs;
  double acc = 0.0;
  const int tid = threadIdx.x;
  for (int base = 0; base < nv; base += kSensThreads * kUnroll) {
    u4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int i = base + u * kSensThreads + tid;
      v[u] = i < nv ? __builtin_nontemporal_load(src + i) : (u4){0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc += sq_vec(v[u], a.dtype);
  }
  for (int d = 32; d >= 1; d >>= 1) acc += __shfl_xor(acc, d, 64);
  __shared__ double wsum[kSensThreads / 64];
  if ((tid & 63) == 0) wsum[tid >> 6] = acc;
  __syncthreads();
  if (tid == 0)
    a.partial[slab * a.chunks + chunk] = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
}

// w[i] = sum over sequences (in order) of the sequence's chunk sums (in
// order), divided by T and by the number of sequences.
__global__ void sens_reduce_kernel(SensLaunch a) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n_comp) return;
  double total = 0.0;
  for (int s = 0; s < a.n_seq; ++s) {
    const double* p = a.partial + ((size_t)s * a.n_comp + i) * a.chunks;
    double seq = 0.0;
    for (int c = 0; c < a.chunks; ++c) seq += p[c];
    total += seq / a.T;
  }
  a.w[i] = total / a.n_seq;
}

}  // namespace

hipError_t launch_sensitivity(const SensLaunch& a, hipStream_t s) {
  dim3 grid(a.chunks, a.n_comp, a.n_seq);
  hipLaunchKernelGGL(sens_kernel, grid, dim3(kSensThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sens_reduce_kernel, dim3((a.n_comp + 255) / 256), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace rq
