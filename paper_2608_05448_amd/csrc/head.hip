// Branch log-probabilities of the DBLast drafter head (Sec. "Architecture": every category
// branch goes through the reused target LM head; q_k(. | y, z) is the softmax of the logits).
//
// bf16 path: logits^T = w * h^T on MFMA (v_mfma_f32_32x32x16_bf16, fp32 accumulation) with the
// vocabulary along the MFMA rows and the branch rows along the MFMA columns, so each lane holds
// 16 logits of one branch row. The per-tile (128 ids) max and sum of exponentials therefore
// reduce in registers plus one cross-half exchange, and the tile-normalised log-probs are
// stored straight from the accumulators: logits never reach memory.
//
// fp32 path: a plain fp32 kernel for fp32 inputs (small problems).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"

namespace dbl {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kVTile = 128;

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Tile configuration of the bf16 head kernel.
//   BV x BM   vocabulary rows x branch rows per workgroup
//   BK        hidden-dimension slice staged in LDS per step (double-buffered)
//   WV x WM   waves; each wave owns a 128 x (BM / WM) block: one full vocabulary tile
template <int BV_, int BM_, int BK_, int WV_, int WM_>
struct HeadCfg {
  static constexpr int BV = BV_, BM = BM_, BK = BK_, WV = WV_, WM = WM_;
  static constexpr int kThreads = WV * WM * 64;
  static constexpr int TM = BM / WM;           // branch rows per wave
  static constexpr int NCB = TM / 32;          // 32-wide MFMA column blocks per wave
  static constexpr int NRB = kVTile / 32;      // 32-high MFMA row blocks per wave (4)
  static constexpr int LDK = BK + 8;           // padded LDS row (bf16 elements)
  static constexpr int CPR = BK / 8;           // 16-byte chunks per row
  static constexpr int A_CHUNKS = BV * CPR / kThreads;
  static constexpr int B_CHUNKS = BM * CPR / kThreads;
  static_assert(BV == WV * kVTile, "each wave owns one vocabulary tile");
  static_assert(TM % 32 == 0, "wave column extent must be a multiple of 32");
  static_assert(BK % 16 == 0, "BK must be a multiple of the MFMA K (16)");
  static_assert((BV * CPR) % kThreads == 0 && (BM * CPR) % kThreads == 0, "even staging");
};

using Cfg = HeadCfg<256, 128, 32, 2, 2>;

// Maps the hardware workgroup id to a logical tile so that consecutive logical tiles (the
// branch-row tiles that share one vocabulary slab of w) land on the same XCD: workgroups are
// dispatched round-robin over the 8 XCDs, each with its own L2.
__device__ __forceinline__ int xcd_remap(int id, int n) {
  const int q = n >> 3, rem = n & 7;
  const int x = id & 7, s = id >> 3;
  return x < rem ? x * (q + 1) + s : rem * (q + 1) + (x - rem) * q + s;
}

template <class C>
__global__ __launch_bounds__(C::kThreads, 2) void head_bf16_kernel(
    const __bf16* __restrict__ h, const __bf16* __restrict__ w, float* __restrict__ tls,
    float* __restrict__ lmass, int64_t M, int64_t V, int d, int nT, int n_mtiles, int vec4) {
  __shared__ __attribute__((aligned(16))) __bf16 As[2][C::BV * C::LDK];
  __shared__ __attribute__((aligned(16))) __bf16 Bs[2][C::BM * C::LDK];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wv = wave / C::WM;  // wave row (vocabulary)
  const int wm = wave % C::WM;  // wave column (branch rows)

  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = logical % n_mtiles;
  const int vt = logical / n_mtiles;
  const int64_t v0 = static_cast<int64_t>(vt) * C::BV;
  const int64_t m0 = static_cast<int64_t>(mt) * C::BM;

  // Staging: thread chunk c -> row c / CPR, 16-byte column c % CPR.
  const __bf16* a_src[C::A_CHUNKS];
  const __bf16* b_src[C::B_CHUNKS];
  int a_dst[C::A_CHUNKS], b_dst[C::B_CHUNKS], a_col[C::A_CHUNKS], b_col[C::B_CHUNKS];
#pragma unroll
  for (int i = 0; i < C::A_CHUNKS; ++i) {
    const int c = tid + i * C::kThreads;
    const int row = c / C::CPR, col = c % C::CPR;
    int64_t gv = v0 + row;
    gv = gv < V ? gv : V - 1;
    a_src[i] = w + gv * d + col * 8;
    a_dst[i] = row * C::LDK + col * 8;
    a_col[i] = col * 8;
  }
#pragma unroll
  for (int i = 0; i < C::B_CHUNKS; ++i) {
    const int c = tid + i * C::kThreads;
    const int row = c / C::CPR, col = c % C::CPR;
    int64_t gm = m0 + row;
    gm = gm < M ? gm : M - 1;
    b_src[i] = h + gm * d + col * 8;
    b_dst[i] = row * C::LDK + col * 8;
    b_col[i] = col * 8;
  }

  u32x4 a_reg[C::A_CHUNKS], b_reg[C::B_CHUNKS];
  auto load_stage = [&](int k0) {
#pragma unroll
    for (int i = 0; i < C::A_CHUNKS; ++i) {
      if (k0 + a_col[i] < d)
        a_reg[i] = *reinterpret_cast<const u32x4*>(a_src[i] + k0);
      else
        a_reg[i] = u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < C::B_CHUNKS; ++i) {
      if (k0 + b_col[i] < d)
        b_reg[i] = *reinterpret_cast<const u32x4*>(b_src[i] + k0);
      else
        b_reg[i] = u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int i = 0; i < C::A_CHUNKS; ++i)
      *reinterpret_cast<u32x4*>(&As[buf][a_dst[i]]) = a_reg[i];
#pragma unroll
    for (int i = 0; i < C::B_CHUNKS; ++i)
      *reinterpret_cast<u32x4*>(&Bs[buf][b_dst[i]]) = b_reg[i];
  };

  f32x16 acc[C::NRB][C::NCB];
#pragma unroll
  for (int rb = 0; rb < C::NRB; ++rb)
#pragma unroll
    for (int cb = 0; cb < C::NCB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[rb][cb][r] = 0.0f;

  const int nk = (d + C::BK - 1) / C::BK;
  load_stage(0);
  store_stage(0);
  __syncthreads();

  const int frag_row = lane & 31;
  const int frag_k = (lane >> 5) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_stage((kt + 1) * C::BK);
#pragma unroll
    for (int kk = 0; kk < C::BK; kk += 16) {
      bf16x8 af[C::NRB], bfr[C::NCB];
#pragma unroll
      for (int rb = 0; rb < C::NRB; ++rb)
        af[rb] = *reinterpret_cast<const bf16x8*>(
            &As[buf][(wv * kVTile + rb * 32 + frag_row) * C::LDK + kk + frag_k]);
#pragma unroll
      for (int cb = 0; cb < C::NCB; ++cb)
        bfr[cb] = *reinterpret_cast<const bf16x8*>(
            &Bs[buf][(wm * C::TM + cb * 32 + frag_row) * C::LDK + kk + frag_k]);
#pragma unroll
      for (int rb = 0; rb < C::NRB; ++rb)
#pragma unroll
        for (int cb = 0; cb < C::NCB; ++cb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[rb], bfr[cb], acc[rb][cb],
                                                                 0, 0, 0);
    }
    if (kt + 1 < nk) store_stage(buf ^ 1);
    __syncthreads();
  }

  // Epilogue: this wave holds the logits of vocabulary tile t for TM branch rows. Lane l holds
  // column (branch row) l % 32 of each 32-column block and, in register r of row block rb,
  // vocabulary id v0w + 32 rb + 8 (r / 4) + 4 (l / 32) + r % 4.
  const int64_t v0w = v0 + wv * kVTile;
  if (v0w >= V) return;
  const int t = static_cast<int>(v0w / kVTile);
  const int half = lane >> 5;
#pragma unroll
  for (int cb = 0; cb < C::NCB; ++cb) {
    const int64_t m = m0 + wm * C::TM + cb * 32 + (lane & 31);
    float mx = -INFINITY;
#pragma unroll
    for (int rb = 0; rb < C::NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t v = v0w + rb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (v < V) mx = fmaxf(mx, acc[rb][cb][r]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    float s = 0.0f;
#pragma unroll
    for (int rb = 0; rb < C::NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t v = v0w + rb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (v < V) s += __expf(acc[rb][cb][r] - mx);
      }
    s += __shfl_xor(s, 32);
    const float lm = mx + __logf(s);
    if (m < M) {
      float* row = tls + m * V;
      if (half == 0) lmass[m * nT + t] = lm;
#pragma unroll
      for (int rb = 0; rb < C::NRB; ++rb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int64_t v = v0w + rb * 32 + 8 * g + 4 * half;
          if (vec4 && v + 3 < V) {
            float4 o;
            o.x = acc[rb][cb][4 * g + 0] - lm;
            o.y = acc[rb][cb][4 * g + 1] - lm;
            o.z = acc[rb][cb][4 * g + 2] - lm;
            o.w = acc[rb][cb][4 * g + 3] - lm;
            *reinterpret_cast<float4*>(row + v) = o;
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (v + e < V) row[v + e] = acc[rb][cb][4 * g + e] - lm;
          }
        }
    }
  }
}

// fp32 path: workgroup (vocabulary tile t, 4 branch rows); thread j owns id 128 t + j.
constexpr int kF32Rows = 4;
constexpr int kF32DChunk = 512;

__global__ __launch_bounds__(128) void head_f32_kernel(const float* __restrict__ h,
                                                       const float* __restrict__ w,
                                                       float* __restrict__ tls,
                                                       float* __restrict__ lmass, int64_t M,
                                                       int64_t V, int d, int nT) {
  __shared__ float hs[kF32Rows][kF32DChunk];
  __shared__ float red[2][kF32Rows];
  const int t = blockIdx.x;
  const int64_t m0 = static_cast<int64_t>(blockIdx.y) * kF32Rows;
  const int j = threadIdx.x;
  const int64_t v = static_cast<int64_t>(t) * kVTile + j;
  const bool valid = v < V;
  float acc[kF32Rows];
#pragma unroll
  for (int r = 0; r < kF32Rows; ++r) acc[r] = 0.0f;
  for (int k0 = 0; k0 < d; k0 += kF32DChunk) {
    const int kn = min(kF32DChunk, d - k0);
    __syncthreads();
    for (int i = j; i < kF32Rows * kF32DChunk; i += 128) {
      const int r = i / kF32DChunk, k = i % kF32DChunk;
      const int64_t m = m0 + r;
      hs[r][k] = (m < M && k < kn) ? h[m * d + k0 + k] : 0.0f;
    }
    __syncthreads();
    if (valid) {
      const float* wr = w + v * d + k0;
      for (int k = 0; k < kn; ++k) {
        const float wk = wr[k];
#pragma unroll
        for (int r = 0; r < kF32Rows; ++r) acc[r] = fmaf(hs[r][k], wk, acc[r]);
      }
    }
  }
  const int wave = j >> 6;
#pragma unroll
  for (int r = 0; r < kF32Rows; ++r) {
    float mx = wave_max(valid ? acc[r] : -INFINITY);
    if ((j & 63) == 0) red[wave][r] = mx;
    __syncthreads();
    mx = fmaxf(red[0][r], red[1][r]);
    __syncthreads();
    float s = wave_sum(valid ? __expf(acc[r] - mx) : 0.0f);
    if ((j & 63) == 0) red[wave][r] = s;
    __syncthreads();
    s = red[0][r] + red[1][r];
    __syncthreads();
    const float lm = mx + __logf(s);
    const int64_t m = m0 + r;
    if (m < M) {
      if (valid) tls[m * V + v] = acc[r] - lm;
      if (j == 0) lmass[m * nT + t] = lm;
    }
  }
}

// lse[m] = log sum_t exp(lmass[m, t]); one wave per row.
__global__ __launch_bounds__(256) void lse_finalize_kernel(const float* __restrict__ lmass,
                                                           float* __restrict__ lse, int64_t M,
                                                           int nT) {
  const int64_t m = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (m >= M) return;
  const float* row = lmass + m * nT;
  float mx = -INFINITY;
  for (int t = lane; t < nT; t += 64) mx = fmaxf(mx, row[t]);
  mx = wave_max(mx);
  float s = 0.0f;
  for (int t = lane; t < nT; t += 64) s += __expf(row[t] - mx);
  s = wave_sum(s);
  if (lane == 0) lse[m] = mx + __logf(s);
}

}  // namespace

hipError_t launch_head(const HeadArgs& a, hipStream_t stream) {
  const int nT = static_cast<int>((a.V + kVTile - 1) / kVTile);
  if (a.dtype_bf16) {
    const int n_mtiles = static_cast<int>((a.M + Cfg::BM - 1) / Cfg::BM);
    const int64_t n_vtiles = (a.V + Cfg::BV - 1) / Cfg::BV;
    const int64_t nwg = n_vtiles * n_mtiles;
    if (nwg > 0x7fffffff) return hipErrorInvalidConfiguration;
    const int vec4 = (a.V % 4 == 0) ? 1 : 0;
    hipLaunchKernelGGL(head_bf16_kernel<Cfg>, dim3(static_cast<unsigned>(nwg)),
                       dim3(Cfg::kThreads), 0, stream, static_cast<const __bf16*>(a.h),
                       static_cast<const __bf16*>(a.w), a.tls, a.lmass, a.M, a.V, a.d, nT,
                       n_mtiles, vec4);
  } else {
    const int64_t mblocks = (a.M + kF32Rows - 1) / kF32Rows;
    if (mblocks > 65535) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(head_f32_kernel, dim3(nT, static_cast<unsigned>(mblocks)), dim3(128), 0,
                       stream, static_cast<const float*>(a.h), static_cast<const float*>(a.w),
                       a.tls, a.lmass, a.M, a.V, a.d, nT);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t lse_blocks = (a.M + 3) / 4;
  hipLaunchKernelGGL(lse_finalize_kernel, dim3(static_cast<unsigned>(lse_blocks)), dim3(256), 0,
                     stream, a.lmass, a.lse, a.M, nT);
  return hipGetLastError();
}

}  // namespace dbl
