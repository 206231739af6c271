// Block draw from the DBLast latent mixture (Sec. "Dependent Block Drafting and Verification":
// draw a category from the prior, then every position of the block in parallel from that
// branch). Two kernels:
//   sample_tiles   grid (position, group of three chunks of 32 vocabulary tiles), 256 threads:
//                  the drawn category's row is streamed once; 8 lanes per 128-id tile each
//                  quantise 16 ids (four 16-byte loads) and the tile's exact integer mass
//                  sum_v floor(q(v) 2^40) goes to the workspace;
//   sample_select  one 256-thread workgroup per position: inverse CDF over the tile sums, then a
//                  scan of the selected tile (the category is read back from z_out).
// The integer masses are quant_detexp32 values (the contract's quant40(detexp32(.)) without its
// branches), summed exactly in binary64: ~30 VALU instructions per vocabulary id.
// Built with floating-point contraction off: every probability that decides a draw follows
// the determinism contract exactly.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "contract.hpp"
#include "kernels.hpp"
#include "wave.hpp"

namespace dbl {
namespace {

// Chunks of 32 tiles per workgroup: every workgroup first waits for its wavefront 0's category
// draw, so three chunks share that wait (18% faster than one at the Qwen3-8B shape, 15% at the
// stress shape; 2, 4, 6 and 8 measured between).
constexpr int kChunksPerGroup = 3;

__global__ __launch_bounds__(256) void sample_tiles_kernel(SampleArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t pos = blockIdx.x;
  const int64_t b = pos / k_.K;
  const int64_t k = pos % k_.K;
  // The block's category: drawn by wavefront 0 alone (every workgroup of the block draws the
  // same one) and shared through LDS.
  __shared__ int s_z;
  if (threadIdx.x < 64) {
    const int zz = draw_category(k_, b);
    if (threadIdx.x == 0) s_z = zz;
  }
  __syncthreads();
  const int z = s_z;
  if (blockIdx.y == 0 && k == 0 && threadIdx.x == 0) a.z_out[b] = z;
  const int sub = threadIdx.x & 7;                     // lane within the tile's group of 8
#pragma unroll 1
  for (int cc = 0; cc < kChunksPerGroup; ++cc) {
    const int t = (blockIdx.y * kChunksPerGroup + cc) * kTilesPerChunk + (threadIdx.x >> 3);
    // The tile's integer mass, summed exactly in binary64 (at most 128 terms below 2^41).
    double s = 0.0;
    if (z >= 0 && t < k_.nT) {
      const int64_t m = (b * k_.K + k) * k_.R + z;
      const float off = __fsub_rn(k_.lmass[m * k_.nT + t], k_.lse[m]);
      const int64_t v0 = static_cast<int64_t>(t) * kTile;
      const float* row = k_.tls + m * k_.V + v0;
      if ((k_.V & 3) == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int v = 4 * sub + 32 * i;
          if (v0 + v < k_.V) {
            // Plain loads: this kernel is bound by VALU issue, and the non-temporal form
            // measured 5% slower here.
            const float4 x = *reinterpret_cast<const float4*>(row + v);
            s += (quant_detexp32_d(__fadd_rn(x.x, off)) + quant_detexp32_d(__fadd_rn(x.y, off))) +
                 (quant_detexp32_d(__fadd_rn(x.z, off)) + quant_detexp32_d(__fadd_rn(x.w, off)));
          }
        }
      } else {
#pragma unroll 4
        for (int i = 0; i < 16; ++i) {
          const int v = sub + 8 * i;
          if (v0 + v < k_.V) s += quant_detexp32_d(__fadd_rn(row[v], off));
        }
      }
    }
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    s += __shfl_xor(s, 4);
    if (sub == 0 && t < k_.nT) a.tilesum[pos * k_.nT + t] = static_cast<uint64_t>(s);
  }
}

__global__ __launch_bounds__(256) void sample_select_kernel(SampleArgs a) {
  __shared__ uint64_t lds[8];
  const BlockArgs& k_ = a.blk;
  const int64_t pos = blockIdx.x;
  const int64_t b = pos / k_.K;
  const int64_t k = pos % k_.K;
  const int z = a.z_out[b];  // the block's category, written by sample_tiles_kernel
  int x = -1;
  if (z >= 0) {
    const int64_t m = (b * k_.K + k) * k_.R + z;
    const float* row = k_.tls + m * k_.V;
    const float* lm = k_.lmass + m * k_.nT;
    const float lse = k_.lse[m];
    const uint32_t r = draw(k_.seed, kToken, static_cast<uint32_t>(k),
                            static_cast<uint64_t>(k_.seq_offset + b), k_.step);
    x = select_by_tiles_block(
        a.tilesum + pos * k_.nT, k_.nT, k_.V, r,
        [&](int64_t v) { return quant_detexp32(__fadd_rn(row[v], __fsub_rn(lm[v / kTile], lse))); },
        lds);
  }
  if (threadIdx.x == 0) a.x_out[b * k_.K + k] = x;
}

}  // namespace

hipError_t launch_sample(const SampleArgs& a, hipStream_t stream) {
  const int64_t npos = a.blk.B * a.blk.K;
  const int nchunk = n_chunks(a.blk.nT);
  if (npos > 0x7fffffff) return hipErrorInvalidConfiguration;
  const int ngroups = (nchunk + kChunksPerGroup - 1) / kChunksPerGroup;
  hipLaunchKernelGGL(sample_tiles_kernel, dim3(static_cast<unsigned>(npos), ngroups), dim3(256),
                     0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sample_select_kernel, dim3(static_cast<unsigned>(npos)), dim3(256), 0,
                     stream, a);
  return hipGetLastError();
}

}  // namespace dbl
