// Block draw from the DBLast latent mixture (Sec. "Dependent Block Drafting and Verification":
// draw a category from the prior, then every position of the block in parallel from that
// branch). One 256-thread workgroup per block position:
//   * wavefront 0 draws the block's category (every position of the block draws the same one);
//   * the token is drawn in two stages on the head's two-level log-probabilities: the 128-id
//     tile by an inverse CDF on floor(detexp32(fl32(lmass_t - lse)) 2^40) over the row's tiles
//     (Philox word 0), then the id within it by an inverse CDF on floor(detexp32(tls_v) 2^40)
//     over the tile's ids (word 1); the product of the two laws is q_k(v | z).
// A position reads its row's ~V / 128 tile masses and one 512-byte tile, not the V-wide row.
// Built with floating-point contraction off: every probability that decides a draw follows
// the determinism contract exactly.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "contract.hpp"
#include "kernels.hpp"
#include "wave.hpp"

namespace dbl {
namespace {

__global__ __launch_bounds__(256) void sample_kernel(SampleArgs a) {
  __shared__ int s_z;
  __shared__ uint64_t lds[8];
  const BlockArgs& k_ = a.blk;
  const int64_t pos = blockIdx.x;
  const int64_t b = pos / k_.K;
  const int64_t k = pos % k_.K;
  if (threadIdx.x < 64) {
    const int zz = draw_category(k_, b);
    if (threadIdx.x == 0) s_z = zz;
  }
  __syncthreads();
  const int z = s_z;  // the same in every thread, so the branches below are uniform
  if (k == 0 && threadIdx.x == 0) a.z_out[b] = z;
  int x = -1;
  if (z >= 0) {
    const int64_t m = (b * k_.K + k) * k_.R + z;
    const float* lm = k_.lmass + m * k_.nT;
    const float lse = k_.lse[m];
    const PhiloxPair r = draw2(k_.seed, kToken, static_cast<uint32_t>(k),
                               static_cast<uint64_t>(k_.seq_offset + b), k_.step);
    const int t = select_block(
        k_.nT, [&](int i) { return lm[i]; },
        [&](float l) { return quant_detexp32(__fsub_rn(l, lse)); }, r.w0, lds);
    if (t >= 0) {
      const int64_t v0 = static_cast<int64_t>(t) * kTile;
      const int n = static_cast<int>(k_.V - v0 < kTile ? k_.V - v0 : kTile);
      const float* tile = k_.tls + m * k_.V + v0;
      const int j = select_block(
          n, [&](int i) { return tile[i]; }, [](float v) { return quant_detexp32(v); }, r.w1, lds);
      if (j >= 0) x = static_cast<int>(v0 + j);
    }
  }
  if (threadIdx.x == 0) a.x_out[b * k_.K + k] = x;
}

}  // namespace

hipError_t launch_sample(const SampleArgs& a, hipStream_t stream) {
  const int64_t npos = a.blk.B * a.blk.K;
  if (npos > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(sample_kernel, dim3(static_cast<unsigned>(npos)), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace dbl
