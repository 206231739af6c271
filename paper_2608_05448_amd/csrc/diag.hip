// Streaming-read probe: the plain read rate that bounds the bandwidth-bound kernels (the
// acceptance-mass stream, the draw's tile sums, the target transform). Every 16-byte word of
// a buffer is read once with 16-byte non-temporal loads (the form those kernels use), four in
// flight per thread; each workgroup writes the sum of what it read, so the loads cannot be
// dropped.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"
#include "wave.hpp"

namespace dbl {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 4;

__global__ __launch_bounds__(kProbeThreads) void read_probe_kernel(const float4* __restrict__ x,
                                                                   int64_t n4,
                                                                   float* __restrict__ part) {
  constexpr int64_t kSpan = static_cast<int64_t>(kProbeThreads) * kProbeUnroll;
  float acc = 0.0f;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kSpan;
  for (int64_t i = blockIdx.x * kSpan + threadIdx.x; i < n4; i += stride) {
    float4 v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) {
      const int64_t j = i + u * kProbeThreads;
      v[u] = j < n4 ? load_stream4(reinterpret_cast<const float*>(x + j))
                    : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    }
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) acc += (v[u].x + v[u].y) + (v[u].z + v[u].w);
  }
  __shared__ float red[kProbeThreads / 64];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

}  // namespace

hipError_t launch_read_probe(const void* buf, int64_t bytes, float* partials, int64_t n_partials,
                             hipStream_t stream) {
  if (n_partials < 1 || n_partials > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(read_probe_kernel, dim3(static_cast<unsigned>(n_partials)),
                     dim3(kProbeThreads), 0, stream, static_cast<const float4*>(buf), bytes / 16,
                     partials);
  return hipGetLastError();
}

}  // namespace dbl
