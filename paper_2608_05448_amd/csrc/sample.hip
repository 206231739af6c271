// Block draw from the DBLast latent mixture (Sec. "Dependent Block Drafting and Verification":
// draw a category from the prior, then every position of the block in parallel from that
// branch). Two kernels:
//   sample_tiles   grid (position, vocabulary chunk): the drawn category's row is streamed
//                  once; each 128-id tile's integer mass sum_v floor(q(v) 2^40) goes to the
//                  workspace;
//   sample_select  one wavefront per position: inverse CDF over the tile sums, then a scan of
//                  the selected tile.
// Built with floating-point contraction off: every probability that decides a draw follows
// the determinism contract exactly.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "contract.hpp"
#include "kernels.hpp"
#include "wave.hpp"

namespace dbl {
namespace {

__global__ __launch_bounds__(256) void sample_tiles_kernel(SampleArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t pos = blockIdx.x;
  const int64_t b = pos / k_.K;
  const int64_t k = pos % k_.K;
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int z = draw_category(k_, b);
  if (blockIdx.y == 0 && k == 0 && threadIdx.x == 0) a.z_out[b] = z;
  uint64_t* out = a.tilesum + pos * k_.nT;
  const int t_begin = blockIdx.y * kTilesPerChunk;
  const int t_end = min(k_.nT, t_begin + kTilesPerChunk);
  if (z < 0) {
    for (int t = t_begin + static_cast<int>(threadIdx.x); t < t_end; t += blockDim.x) out[t] = 0;
    return;
  }
  const int64_t m = (b * k_.K + k) * k_.R + z;
  const float* row = k_.tls + m * k_.V;
  const float lse = k_.lse[m];
  for (int t = t_begin + wave; t < t_end; t += 4) {
    const float off = __fsub_rn(k_.lmass[m * k_.nT + t], lse);
    const int64_t v = static_cast<int64_t>(t) * kTile + 2 * lane;
    uint64_t s = 0;
    if (v < k_.V) s += quant40(detexp32(__fadd_rn(row[v], off)));
    if (v + 1 < k_.V) s += quant40(detexp32(__fadd_rn(row[v + 1], off)));
    s = wave_sum_u64(s);
    if (lane == 0) out[t] = s;
  }
}

__global__ __launch_bounds__(64) void sample_select_kernel(SampleArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t pos = blockIdx.x;
  const int64_t b = pos / k_.K;
  const int64_t k = pos % k_.K;
  const int z = draw_category(k_, b);
  int x = -1;
  if (z >= 0) {
    const int64_t m = (b * k_.K + k) * k_.R + z;
    const float* row = k_.tls + m * k_.V;
    const float* lm = k_.lmass + m * k_.nT;
    const float lse = k_.lse[m];
    const uint32_t r = draw(k_.seed, kToken, static_cast<uint32_t>(k),
                            static_cast<uint64_t>(k_.seq_offset + b), k_.step);
    x = select_by_tiles(a.tilesum + pos * k_.nT, k_.nT, k_.V, r, [&](int64_t v) {
      const float off = __fsub_rn(lm[v / kTile], lse);
      return quant40(detexp32(__fadd_rn(row[v], off)));
    });
  }
  if (threadIdx.x == 0) a.x_out[b * k_.K + k] = x;
}

}  // namespace

hipError_t launch_sample(const SampleArgs& a, hipStream_t stream) {
  const int64_t npos = a.blk.B * a.blk.K;
  const int nchunk = n_chunks(a.blk.nT);
  if (npos > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(sample_tiles_kernel, dim3(static_cast<unsigned>(npos), nchunk), dim3(256),
                     0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sample_select_kernel, dim3(static_cast<unsigned>(npos)), dim3(64), 0,
                     stream, a);
  return hipGetLastError();
}

}  // namespace dbl
