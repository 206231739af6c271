// Test helper (not part of the library): checks on the GPU, for every one of the 2^32 binary32
// bit patterns, that the branch-free quantised exponential the sampler and verifier use equals the
// determinism contract's definition quant40(detexp32(x)) = floor(detexp32(x) 2^40).
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

}  // namespace

// bad: device u64, zeroed by the caller; first: device u32, set to 0xffffffff by the caller.
extern "C" int dbl_test_quant_exhaustive(unsigned long long* bad, unsigned* first, void* stream) {
  const unsigned blocks = static_cast<unsigned>((uint64_t(1) << 32) / (256 * kPerThread));
  hipLaunchKernelGGL(quant_all_kernel, dim3(blocks), dim3(256), 0,
                     static_cast<hipStream_t>(stream), bad, first);
  return static_cast<int>(hipGetLastError());
}
