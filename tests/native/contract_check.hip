// Test helper (not part of the library): checks on the GPU, for every one of the 2^32 binary32
// bit patterns, that the branch-free quantised exponential the sampler and verifier use equals the
// determinism contract's definition quant40(detexp32(x)) = floor(detexp32(x) 2^40); and evaluates
// the kernels' Philox4x32-10 (output words 0 and 1) on given counters and keys.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../paper_2608_05448_amd/csrc/contract.hpp"

namespace {

constexpr int kPerThread = 256;

__global__ __launch_bounds__(256) void quant_all_kernel(unsigned long long* bad, unsigned* first) {
  const uint64_t u0 = (static_cast<uint64_t>(blockIdx.x) * 256 + threadIdx.x) * kPerThread;
  unsigned long long nbad = 0;
  unsigned fb = 0xffffffffu;
  for (int i = 0; i < kPerThread; ++i) {
    const uint32_t u = static_cast<uint32_t>(u0 + i);
    const float x = __uint_as_float(u);
    const uint64_t ref = dbl::quant40(dbl::detexp32(x));
    const uint64_t a = dbl::quant_detexp32(x);
    if (a != ref) {
      ++nbad;
      fb = fb < u ? fb : u;
    }
  }
  if (nbad) {
    atomicAdd(bad, nbad);
    atomicMin(first, fb);
  }
}

__global__ __launch_bounds__(64) void philox01_kernel(const uint32_t* in, uint32_t* out, int n) {
  const int i = blockIdx.x * 64 + threadIdx.x;
  if (i >= n) return;
  const uint32_t* w = in + 6 * i;
  const dbl::PhiloxPair r = dbl::philox_words01(w[0], w[1], w[2], w[3], w[4], w[5]);
  out[2 * i] = r.w0;
  out[2 * i + 1] = r.w1;
}

}  // namespace

// in: device [n, 6] u32 (counter words 0..3, key words 0..1); out: device [n, 2] u32.
extern "C" int dbl_test_philox01(const uint32_t* in, uint32_t* out, int n, void* stream) {
  if (n <= 0) return 0;
  hipLaunchKernelGGL(philox01_kernel, dim3((n + 63) / 64), dim3(64), 0,
                     static_cast<hipStream_t>(stream), in, out, n);
  return static_cast<int>(hipGetLastError());
}

// bad: device u64, zeroed by the caller; first: device u32, set to 0xffffffff by the caller.
extern "C" int dbl_test_quant_exhaustive(unsigned long long* bad, unsigned* first, void* stream) {
  const unsigned blocks = static_cast<unsigned>((uint64_t(1) << 32) / (256 * kPerThread));
  hipLaunchKernelGGL(quant_all_kernel, dim3(blocks), dim3(256), 0,
                     static_cast<hipStream_t>(stream), bad, first);
  return static_cast<int>(hipGetLastError());
}
