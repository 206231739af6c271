// Branch log-probabilities of the DBLast drafter head (Sec. "Architecture": every category
// branch goes through the reused target LM head; q_k(. | y, z) is the softmax of the logits).
//
// bf16 path: logits^T = w * h^T on MFMA (v_mfma_f32_32x32x16_bf16, fp32 accumulation) with the
// vocabulary along the MFMA rows and the branch rows along the MFMA columns, so each lane holds
// 16 logits of one branch row. The per-tile (128 ids) max and sum of exponentials therefore
// reduce in registers plus one cross-half exchange, and the tile-normalised log-probs are
// stored straight from the accumulators: logits never reach memory. Operand feeds, by hidden
// size: d % 64 == 0, the 8-wave ping-pong kernel with 64-deep stages copied global -> LDS
// directly (the main path); d % 32 == 0, 32-deep stages copied global -> LDS by four waves;
// otherwise a register-staged kernel with padded LDS rows. The branch expander runs a
// register-staged kernel with 64-deep stages and 128 x 256 tiles.
//
// fp32 path: a plain fp32 kernel for fp32 inputs (small problems).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "kernels.hpp"

namespace dbl {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kVTile = 128;
constexpr float kLog2e = 1.4426950408889634f;

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

// Argmax of a row across vocabulary tiles: every tile contributes the 64-bit key
// (order-preserving bits of its maximum logit, ~id) through an atomic maximum, so the winner is
// the largest logit and, among equal logits, the lowest id. -0 is folded into +0.
__device__ __forceinline__ uint64_t argmax_key(float x, int64_t v) {
  uint32_t u = __float_as_uint(x + 0.0f);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<uint64_t>(u) << 32) | (0xFFFFFFFFu - static_cast<uint32_t>(v));
}

// Epilogue shared by the bf16 kernels. The wave holds the logits of one vocabulary tile (ids
// v0w .. v0w + 127) for NCB * 32 branch rows. Lane l holds row m0w + 32 cb + l % 32 and, in
// register r of row block rb, id v0w + 32 rb + 8 (r / 4) + 4 (l / 32) + r % 4. For each row:
// tile max and sum of exponentials in registers plus one cross-half exchange, then the tile
// log-mass and the tile-normalised log-probs are written; logits never reach memory.
template <int NRB, int NCB, bool ARG>
__device__ __forceinline__ void tile_logsoftmax_store(f32x16 (&acc)[NRB][NCB], float* tls,
                                                      float* lmass, uint64_t* amax, int64_t M,
                                                      int64_t V, int nT, int64_t v0w,
                                                      int64_t m0w, int lane, int vec4) {
  const int half = lane >> 5;
  const int t = static_cast<int>(v0w / kVTile);
  const int vlim = static_cast<int>(V - v0w < kVTile ? V - v0w : kVTile);  // ids in this tile
  const bool full = vlim == kVTile;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    const int64_t m = m0w + cb * 32 + (lane & 31);
    float mx = -INFINITY;
    float s = 0.0f;
    int vi = 0;  // offset in the tile of this lane's first maximum (ARG only)
    if (full) {
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, acc[rb][cb][r]);
      if constexpr (ARG) {  // this lane's first id holding its maximum (ids rise with rb, r)
        vi = 1 << 30;
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (acc[rb][cb][r] == mx) vi = min(vi, rb * 32 + 8 * (r >> 2) + 4 * half + (r & 3));
        vi = vi == (1 << 30) ? 0 : vi;
        const float omx = __shfl_xor(mx, 32);
        const int ovi = __shfl_xor(vi, 32);
        if (omx > mx || (omx == mx && ovi < vi)) {
          mx = omx;
          vi = ovi;
        }
      } else {
        mx = fmaxf(mx, __shfl_xor(mx, 32));
      }
      const float nb = -mx * kLog2e;
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += __builtin_amdgcn_exp2f(fmaf(acc[rb][cb][r], kLog2e, nb));
    } else {
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int o = rb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          if (o < vlim) mx = fmaxf(mx, acc[rb][cb][r]);
        }
      if constexpr (ARG) {
        vi = 1 << 30;
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int o = rb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
            if (o < vlim && acc[rb][cb][r] == mx) vi = min(vi, o);
          }
        vi = vi == (1 << 30) ? 0 : vi;
        const float omx = __shfl_xor(mx, 32);
        const int ovi = __shfl_xor(vi, 32);
        if (omx > mx || (omx == mx && ovi < vi)) {
          mx = omx;
          vi = ovi;
        }
      } else {
        mx = fmaxf(mx, __shfl_xor(mx, 32));
      }
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (rb * 32 + 8 * (r >> 2) + 4 * half + (r & 3) < vlim)
            s += __expf(acc[rb][cb][r] - mx);
    }
    s += __shfl_xor(s, 32);
    const float lm = mx + __logf(s);
    if (m < M) {
      if (half == 0) lmass[m * nT + t] = lm;
      if constexpr (ARG) {
        if (half == 0) atomicMax(reinterpret_cast<unsigned long long*>(amax + m),
                                 static_cast<unsigned long long>(argmax_key(mx, v0w + vi)));
      }
      float* row = tls + m * V + v0w + 4 * half;
      if (full && vec4) {
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            float4 o;
            o.x = acc[rb][cb][4 * g + 0] - lm;
            o.y = acc[rb][cb][4 * g + 1] - lm;
            o.z = acc[rb][cb][4 * g + 2] - lm;
            o.w = acc[rb][cb][4 * g + 3] - lm;
            *reinterpret_cast<float4*>(row + rb * 32 + 8 * g) = o;
          }
      } else {
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
          for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (rb * 32 + 8 * g + 4 * half + e < vlim)
                row[rb * 32 + 8 * g + e] = acc[rb][cb][4 * g + e] - lm;
      }
    }
  }
}

// Epilogue of the register-staged kernel: the same results as tile_logsoftmax_store, with
// the stores routed through a 16 KB LDS scratch per wave (xp). In the register layout a
// 16-byte store instruction covers 32 rows, 32 bytes each; every row of tls is V * 4 bytes from
// the next, so each such instruction needs tens of address translations, which the vector L1
// serialises. Here the wave writes its 32 rows x 128 ids to LDS as 512-byte rows (16-byte chunk
// c of row r at chunk c ^ (r % 16): conflict-free both ways) and reads them back so that each
// store instruction writes two whole 512-byte row segments. One block of 32 rows at a time:
// its 64 logits per lane are copied out of the accumulators once; in the vocabulary's last,
// partial tile the ids past V are set to -inf first, so every tile takes the same arithmetic.
template <int NRB, int NCB, bool ARG>
__device__ __forceinline__ void tile_logsoftmax_store_lds(f32x16 (&acc)[NRB][NCB], float* tls,
                                                          float* lmass, uint64_t* amax,
                                                          int64_t M, int64_t V, int nT,
                                                          int64_t v0w, int64_t m0w, int lane,
                                                          int vec4, char* xp) {
  const int half = lane >> 5;
  const int lr = lane & 31;
  const int t = static_cast<int>(v0w / kVTile);
  const int vlim = static_cast<int>(V - v0w < kVTile ? V - v0w : kVTile);  // ids in this tile
  const bool full = vlim == kVTile;
  constexpr int NX = NRB * 16;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    __builtin_amdgcn_sched_barrier(0);
    const int64_t m = m0w + cb * 32 + lr;
    float x[NX];  // x[16 rb + r]: id 32 rb + 8 (r / 4) + 4 half + r % 4 of the tile
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int r = 0; r < 16; ++r) x[16 * rb + r] = acc[rb][cb][r];
    // Id offset of x[16 rb + r] in the tile: 32 rb + 8 (r / 4) + (r % 4) + 4 half; the
    // compile-time part is compared against limits shifted by 4 half, so no per-value offset
    // is held in a register.
    if (!full) {
      const int lim = vlim - 4 * half;
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (rb * 32 + 8 * (r >> 2) + (r & 3) >= lim) x[16 * rb + r] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < NX; ++i) mx = fmaxf(mx, x[i]);
    int vi = 0;  // offset in the tile of this lane's first maximum (ARG only)
    if constexpr (ARG) {
      vi = 1 << 30;
#pragma unroll
      for (int rb = NRB - 1; rb >= 0; --rb)
#pragma unroll
        for (int r = 15; r >= 0; --r)
          vi = x[16 * rb + r] == mx ? rb * 32 + 8 * (r >> 2) + (r & 3) : vi;
      vi = vi == (1 << 30) ? 0 : vi + 4 * half;
      const float omx = __shfl_xor(mx, 32);
      const int ovi = __shfl_xor(vi, 32);
      if (omx > mx || (omx == mx && ovi < vi)) {
        mx = omx;
        vi = ovi;
      }
    } else {
      mx = fmaxf(mx, __shfl_xor(mx, 32));
    }
    const float nb = -mx * kLog2e;
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < NX; ++i) s += __builtin_amdgcn_exp2f(fmaf(x[i], kLog2e, nb));
    s += __shfl_xor(s, 32);
    const float lm = mx + __logf(s);
    if (m < M && half == 0) {
      lmass[m * nT + t] = lm;
      if constexpr (ARG)
        atomicMax(reinterpret_cast<unsigned long long*>(amax + m),
                  static_cast<unsigned long long>(argmax_key(mx, v0w + vi)));
    }
    float* const base = tls + (m0w + cb * 32) * V + v0w;  // wave-uniform
    const bool fast = full && vec4 && m0w + cb * 32 + 32 <= M && V < (int64_t{1} << 25);
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float4 o;
        o.x = x[16 * rb + 4 * g + 0] - lm;
        o.y = x[16 * rb + 4 * g + 1] - lm;
        o.z = x[16 * rb + 4 * g + 2] - lm;
        o.w = x[16 * rb + 4 * g + 3] - lm;
        const int chunk = (rb * 8 + 2 * g + half) ^ (lr & 15);
        *reinterpret_cast<float4*>(xp + lr * 512 + chunk * 16) = o;
      }
    // Wave-private LDS region: the writes above precede these reads in the wave's LDS queue.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    float4 o[16];  // o[jj]: ids 4 lr .. 4 lr + 3 of block row 2 jj + half
#pragma unroll
    for (int jj = 0; jj < 16; ++jj) {
      const int rr = 2 * jj + half;
      o[jj] = *reinterpret_cast<const float4*>(xp + rr * 512 + ((lr ^ (rr & 15)) * 16));
    }
    if (fast) {
      const uint32_t lo = static_cast<uint32_t>(half * V + 4 * lr);  // 32-bit lane offsets
      const uint32_t step = static_cast<uint32_t>(2 * V);
#pragma unroll
      // Non-temporal: the 256 KB a workgroup writes per tile would otherwise evict the operand
      // slabs its XCD's other tiles are still reading from L2 (1% faster).
      for (int jj = 0; jj < 16; ++jj)
        __builtin_nontemporal_store(f32x4{o[jj].x, o[jj].y, o[jj].z, o[jj].w},
                                    reinterpret_cast<f32x4*>(base + (lo + jj * step)));
    } else {
#pragma unroll
      for (int jj = 0; jj < 16; ++jj) {
        const int rr = 2 * jj + half;
        if (m0w + cb * 32 + rr < M) {
          float* q = base + rr * V + 4 * lr;
          if (vec4 && 4 * lr + 3 < vlim) {
            *reinterpret_cast<float4*>(q) = o[jj];
          } else {
            if (4 * lr + 0 < vlim) q[0] = o[jj].x;
            if (4 * lr + 1 < vlim) q[1] = o[jj].y;
            if (4 * lr + 2 < vlim) q[2] = o[jj].z;
            if (4 * lr + 3 < vlim) q[3] = o[jj].w;
          }
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
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

using Cfg = HeadCfg<256, 256, 64, 2, 2>;

// Maps the hardware workgroup id to a logical tile id so that consecutive logical ids land on
// the same XCD: workgroups are dispatched round-robin over the 8 XCDs, each with its own L2.
__device__ __forceinline__ int xcd_remap(int id, int n) {
  const int q = n >> 3, rem = n & 7;
  const int x = id & 7, s = id >> 3;
  return x < rem ? x * (q + 1) + s : rem * (q + 1) + (x - rem) * q + s;
}

// Logical tile id -> (vocabulary tile, branch-row tile). Branch-row tiles are taken in groups
// of up to g; a group sweeps every vocabulary tile before the next group starts, and within a
// vocabulary tile the group's branch-row tiles are consecutive. With groups of 4, the ~32
// workgroups resident on one XCD cover about 8 vocabulary x 4 branch-row tiles: each slab of w
// is read by up to 4 of them and each slab of h by about 8, from that XCD's L2. Measured: groups
// of 4 are 1% faster than 8 at 8 branch-row tiles (the Qwen3-8B head) and 1.7% at 32 (B = 256,
// K = 8, R = 4), 3% faster than no grouping; with 128 branch-row tiles (a 128-block chunk at
// K = R = 16, where each group re-streams all of w from HBM) groups of 8 are 1.7% faster than 4
// and groups of 16 or 32 slower.
constexpr int kGroupM = 4;
constexpr int kGroupMLarge = 8;      // from kGroupLargeFrom branch-row tiles up
constexpr int kGroupLargeFrom = 64;
__device__ __forceinline__ void tile_of(int L, int n_vtiles, int n_mtiles, int* vt, int* mt) {
  const int gm = n_mtiles >= kGroupLargeFrom ? kGroupMLarge : kGroupM;
  const int n_groups = (n_mtiles + gm - 1) / gm;
  const int per_full = n_vtiles * gm;
  if (L < (n_groups - 1) * per_full) {
    const int g = L / per_full, rem = L % per_full;
    *vt = rem / gm;
    *mt = g * gm + rem % gm;
  } else {
    const int rem = L - (n_groups - 1) * per_full;
    const int gl = n_mtiles - (n_groups - 1) * gm;
    *vt = rem / gl;
    *mt = (n_groups - 1) * gm + rem % gl;
  }
}

template <class C, bool ARG>
__global__ __launch_bounds__(C::kThreads, 1) void head_bf16_kernel(
    const __bf16* __restrict__ h, const __bf16* __restrict__ w, float* __restrict__ tls,
    float* __restrict__ lmass, uint64_t* __restrict__ amax, int64_t M, int64_t V, int d, int nT,
    int n_mtiles, int vec4) {
  __shared__ __attribute__((aligned(16))) __bf16 As[2][C::BV * C::LDK];
  __shared__ __attribute__((aligned(16))) __bf16 Bs[2][C::BM * C::LDK];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wv = wave / C::WM;  // wave row (vocabulary)
  const int wm = wave % C::WM;  // wave column (branch rows)

  int vt, mt;
  tile_of(xcd_remap(blockIdx.x, gridDim.x), gridDim.x / n_mtiles, n_mtiles, &vt, &mt);
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
  // Global -> registers for the stage at k0. Full stages load unconditionally; the last,
  // partial stage zero-fills the 16-byte chunks beyond d (d % 8 == 0).
  auto load_stage = [&](int k0) {
    if (k0 + C::BK <= d) {
#pragma unroll
      for (int i = 0; i < C::A_CHUNKS; ++i)
        a_reg[i] = *reinterpret_cast<const u32x4*>(a_src[i] + k0);
#pragma unroll
      for (int i = 0; i < C::B_CHUNKS; ++i)
        b_reg[i] = *reinterpret_cast<const u32x4*>(b_src[i] + k0);
    } else {
#pragma unroll
      for (int i = 0; i < C::A_CHUNKS; ++i)
        a_reg[i] = k0 + a_col[i] < d ? *reinterpret_cast<const u32x4*>(a_src[i] + k0)
                                     : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int i = 0; i < C::B_CHUNKS; ++i)
        b_reg[i] = k0 + b_col[i] < d ? *reinterpret_cast<const u32x4*>(b_src[i] + k0)
                                     : u32x4{0u, 0u, 0u, 0u};
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

  // MFMA operand fragments: lane l reads row l % 32 of a 32-row block and the 8 consecutive
  // k values starting at 8 (l / 32) of the current 16-wide k step.
  const int frag_row = lane & 31;
  const int frag_k = (lane >> 5) * 8;
  const int a_frag = (wv * kVTile + frag_row) * C::LDK + frag_k;
  const int b_frag = (wm * C::TM + frag_row) * C::LDK + frag_k;
  bf16x8 af[2][C::NRB], bfr[2][C::NCB];
  auto load_frags = [&](int set, int buf, int kk) {
#pragma unroll
    for (int rb = 0; rb < C::NRB; ++rb)
      af[set][rb] = *reinterpret_cast<const bf16x8*>(&As[buf][a_frag + rb * 32 * C::LDK + kk]);
#pragma unroll
    for (int cb = 0; cb < C::NCB; ++cb)
      bfr[set][cb] = *reinterpret_cast<const bf16x8*>(&Bs[buf][b_frag + cb * 32 * C::LDK + kk]);
  };

  constexpr int KSTEPS = C::BK / 16;
  const int nk = (d + C::BK - 1) / C::BK;
  load_stage(0);
  store_stage(0);
  __syncthreads();
  load_frags(0, 0, 0);

  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) load_stage((kt + 1) * C::BK);
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      const int cur = ks & 1;
      // Fetch the next k step's fragments while this step's MFMAs run.
      if (ks + 1 < KSTEPS) load_frags(cur ^ 1, buf, (ks + 1) * 16);
#pragma unroll
      for (int rb = 0; rb < C::NRB; ++rb)
#pragma unroll
        for (int cb = 0; cb < C::NCB; ++cb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][rb], bfr[cur][cb],
                                                                 acc[rb][cb], 0, 0, 0);
    }
    if (more) store_stage(buf ^ 1);
    __syncthreads();
    if (more) load_frags(0, buf ^ 1, 0);
  }

  const int64_t v0w = v0 + wv * kVTile;
  if (v0w >= V) return;
  tile_logsoftmax_store<C::NRB, C::NCB, ARG>(acc, tls, lmass, amax, M, V, nT, v0w,
                                             m0 + wm * C::TM, lane, vec4);
}

// ---------------------------------------------------------------------------------------
// Direct-to-LDS variant (hidden sizes that are a multiple of BK): operand tiles are copied
// global -> LDS by global_load_lds_dwordx4 into an S-stage ring, issued S - 1 stages ahead, so
// no staging registers are needed and global latency is covered by S - 1 stages of MFMA work.
// LDS rows hold BK bf16; the 16-byte chunks of row r are XOR-permuted by swz(r) so that the
// MFMA fragment reads are free of bank conflicts: ds_read_b128 serves 16 consecutive lanes per
// cycle from 64 four-byte banks (256 B), so rows r, r + 4, r + 8, r + 12 of a 64-byte-row tile
// must land their chunk in different 16-byte bank groups (measured with SQ_LDS_BANK_CONFLICT).
template <int BK_, int S_, int BM_, int WM_>
struct DmaCfg {
  static constexpr int BV = 256, BM = BM_, BK = BK_, S = S_;
  // Waves: 2 along the vocabulary (one 128-id tile each) times WM along the branch rows.
  static constexpr int WM = WM_, NW = 2 * WM, kThreads = 64 * NW;
  static constexpr int TM = BM / WM, NCB = TM / 32, NRB = 4;
  static constexpr int CPR = BK / 8;                     // 16-byte chunks per row
  static constexpr int ROWB = BK * 2;                    // bytes per LDS row
  static constexpr int RPI = 64 / CPR;                   // rows per DMA instruction
  static constexpr int A_INST = BV / RPI / NW;           // DMA instructions per wave, w rows
  static constexpr int B_INST = BM / RPI / NW;           // DMA instructions per wave, h rows
  static constexpr int PER_STAGE = A_INST + B_INST;      // DMA instructions per wave per stage
  static constexpr int TBA = BV * ROWB;                  // bytes of the w tile of one stage
  static constexpr int TBB = BM * ROWB;                  // bytes of the h tile of one stage
  // co-resident workgroups per CU (LDS-limited)
  static constexpr int kWgPerCu = 2 * S * (TBA + TBB) <= 160 * 1024 ? 2 : 1;
  static_assert(CPR == 4 || CPR == 8, "BK must be 32 or 64");
  static_assert(BM == 128 || BM == 256, "branch-row tile of 128 or 256");
  static_assert(WM == 2 || WM == 4, "2 or 4 waves along the branch rows");
  static_assert(TM % 32 == 0 && A_INST >= 1 && B_INST >= 1, "wave tiling");
  static_assert(S >= 2 && S <= 5, "2 to 5 stages");
  static_assert((S - 2) * PER_STAGE <= 63, "vmcnt range");
  static_assert(S * (TBA + TBB) * kWgPerCu <= 160 * 1024, "LDS per CU");
};

template <int CPR>
__device__ __forceinline__ int dma_swz(int r) {
  return CPR == 4 ? ((r >> 2) & 3) : ((r >> 1) & 7);
}

// One global_load_lds_dwordx4: lane i copies 16 bytes from sbase + voff (its own offset) to
// LDS byte M0 + 16 i. Issued through inline asm so that the compiler does not model the LDS write: its
// conservative wait-count insertion would otherwise drain every outstanding stage before each
// LDS read. Completion is tracked explicitly with wait_vmcnt.
__device__ __forceinline__ void lds_dma16(const char* sbase, uint32_t voff, uint32_t m0v) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "{m0}"(m0v)
               : "memory");
}

// LDS byte address of a __shared__ location (the value M0 expects).
__device__ __forceinline__ uint32_t lds_addr(const char* p) {
  return static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) char*)(p)));
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

#ifndef DBL_HEAD_XP
#define DBL_HEAD_XP 1
#endif
#ifndef DBL_HEAD_BK
#define DBL_HEAD_BK 32
#endif
#ifndef DBL_HEAD_STAGES
#define DBL_HEAD_STAGES 4
#endif
#ifndef DBL_HEAD_FRAG_SLOTS
#define DBL_HEAD_FRAG_SLOTS 8
#endif
#ifndef DBL_HEAD_BM
#define DBL_HEAD_BM 256
#endif
#ifndef DBL_HEAD_WM
#define DBL_HEAD_WM 2
#endif
using DCfg = DmaCfg<DBL_HEAD_BK, DBL_HEAD_STAGES, DBL_HEAD_BM, DBL_HEAD_WM>;

// What the direct-to-LDS GEMM does with its accumulators (rows of w on the MFMA rows, rows of h
// on the columns): the head's tile log-softmax (with or without the argmax keys), or the
// category expander's branch states.
enum EpiKind : int { kEpiLogSoftmax = 0, kEpiLogSoftmaxArgmax = 1, kEpiExpand = 2 };

struct EpiArgs {
  float* tls;            // head: [M, V]
  float* lmass;          // head: [M, nT]
  uint64_t* amax;        // head: [M] argmax keys (argmax epilogue)
  int nT, vec4;
  __bf16* out;           // expander: [M, V] branch states, V = R * d
  const __bf16* bias;    // expander: [V]
  const __bf16* hres;    // expander: [M, d] trunk states (the residual)
  int dres;              // expander: d
};

// Expander epilogue: out[m, v] = bf16(h[m, v mod d] + (acc + c[v])), i.e. h_{k,z} = h_k + g_z(h_k)
// with g_z(h) = W_z h + c_z evaluated in fp32 and rounded once. Lane l holds row
// m0w + 32 cb + l % 32 and, in registers 4g..4g+3 of row block rb, the four consecutive features
// v0w + 32 rb + 8 g + 4 (l / 32) + {0..3}, which are stored as one 8-byte write.
template <int NRB, int NCB>
__device__ __forceinline__ void expand_store(f32x16 (&acc)[NRB][NCB], const EpiArgs& e,
                                             int64_t M, int64_t V, int64_t v0w, int64_t m0w,
                                             int lane) {
  const int half = lane >> 5;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    const int64_t m = m0w + cb * 32 + (lane & 31);
    if (m >= M) continue;
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int64_t v = v0w + 32 * rb + 8 * g + 4 * half;
        if (v >= V) continue;
        const int64_t j = v % e.dres;
        const __bf16* hr = e.hres + m * e.dres + j;
        __bf16* o = e.out + m * V + v;
        if (v + 3 < V) {
          typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
          const bf16x4 c4 = *reinterpret_cast<const bf16x4*>(e.bias + v);
          const bf16x4 h4 = *reinterpret_cast<const bf16x4*>(hr);
          bf16x4 y;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            y[q] = static_cast<__bf16>(static_cast<float>(h4[q]) +
                                       (acc[rb][cb][4 * g + q] + static_cast<float>(c4[q])));
          *reinterpret_cast<bf16x4*>(o) = y;
        } else {
          for (int q = 0; q < 4 && v + q < V; ++q)
            o[q] = static_cast<__bf16>(static_cast<float>(hr[q]) +
                                       (acc[rb][cb][4 * g + q] + static_cast<float>(e.bias[v + q])));
        }
      }
  }
}

template <class C, int EPI>
__global__ __launch_bounds__(C::kThreads, C::kWgPerCu) void head_bf16_dma_kernel(
    const __bf16* __restrict__ h, const __bf16* __restrict__ w, const EpiArgs ea, int64_t M,
    int64_t V, int d, int n_mtiles) {
  constexpr int TA = C::TBA, TB = C::TBB;
  __shared__ __attribute__((aligned(1024))) char sA0[TA], sB0[TB], sA1[TA], sB1[TB];
  __shared__ __attribute__((aligned(1024))) char sA2[C::S > 2 ? TA : 16], sB2[C::S > 2 ? TB : 16];
  __shared__ __attribute__((aligned(1024))) char sA3[C::S > 3 ? TA : 16], sB3[C::S > 3 ? TB : 16];
  __shared__ __attribute__((aligned(1024))) char sA4[C::S > 4 ? TA : 16], sB4[C::S > 4 ? TB : 16];
  char* const sA[5] = {sA0, sA1, sA2, sA3, sA4};
  char* const sB[5] = {sB0, sB1, sB2, sB3, sB4};

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar address math
  const int wv = wave / C::WM;
  const int wm = wave % C::WM;

  int vt, mt;
  tile_of(xcd_remap(blockIdx.x, gridDim.x), gridDim.x / n_mtiles, n_mtiles, &vt, &mt);
  const int64_t v0 = static_cast<int64_t>(vt) * C::BV;
  const int64_t m0 = static_cast<int64_t>(mt) * C::BM;

  // DMA sources: instruction i of this wave covers tile rows (wave * INST + i) * RPI + [0, RPI);
  // lane -> row lane / CPR of it and the chunk whose permuted slot is lane % CPR. Addresses are
  // a scalar tile base plus a 32-bit per-lane byte offset (rows past V or M are clamped).
  const char* a_tile = reinterpret_cast<const char*>(w + v0 * d);
  const char* b_tile = reinterpret_cast<const char*>(h + m0 * d);
  uint32_t a_off[C::A_INST], b_off[C::B_INST];
#pragma unroll
  for (int i = 0; i < C::A_INST; ++i) {
    const int r = (wave * C::A_INST + i) * C::RPI + lane / C::CPR;
    const int c = (lane % C::CPR) ^ dma_swz<C::CPR>(r);
    const int64_t gv = v0 + r < V ? r : V - 1 - v0;
    a_off[i] = static_cast<uint32_t>(gv * d * 2 + c * 16);
  }
#pragma unroll
  for (int i = 0; i < C::B_INST; ++i) {
    const int r = (wave * C::B_INST + i) * C::RPI + lane / C::CPR;
    const int c = (lane % C::CPR) ^ dma_swz<C::CPR>(r);
    const int64_t gm = m0 + r < M ? r : M - 1 - m0;
    b_off[i] = static_cast<uint32_t>(gm * d * 2 + c * 16);
  }

  f32x16 acc[C::NRB][C::NCB];
#pragma unroll
  for (int rb = 0; rb < C::NRB; ++rb)
#pragma unroll
    for (int cb = 0; cb < C::NCB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[rb][cb][r] = 0.0f;

  // Fragment addressing: row = block base + lane % 32, chunk (2 ks + lane / 32) ^ swz(row);
  // swz(row) depends on row % 32 = lane % 32 only (block bases are multiples of 32), so the
  // per-k-step offset is a XOR with 32 ks.
  const int tt = 16 * ((lane >> 5) ^ dma_swz<C::CPR>(lane & 31));
  const int a_base = (wv * kVTile + (lane & 31)) * C::ROWB;
  const int b_base = (wm * C::TM + (lane & 31)) * C::ROWB;
  bf16x8 af[2][C::NRB], bfr[2][C::NCB];
  // Fragment i of a k step: i < NRB is A block i, else B block i - NRB.
  auto load_frag = [&](int set, const char* As, const char* Bs, int ks, int i) {
    const int x = (32 * ks) ^ tt;
    if (i < C::NRB)
      af[set][i] = *reinterpret_cast<const bf16x8*>(As + a_base + i * 32 * C::ROWB + x);
    else
      bfr[set][i - C::NRB] =
          *reinterpret_cast<const bf16x8*>(Bs + b_base + (i - C::NRB) * 32 * C::ROWB + x);
  };
  auto mfma = [&](int set, int q) {
    const int rb = q / C::NCB, cb = q % C::NCB;
    acc[rb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[set][rb], bfr[set][cb], acc[rb][cb],
                                                           0, 0, 0);
  };
  auto issue_one = [&](auto slot_c, int k0, int i) {
    constexpr int slot = decltype(slot_c)::value;
    if (i < C::A_INST)
      lds_dma16(a_tile + 2 * k0, a_off[i], lds_addr(sA[slot]) + (wave * C::A_INST + i) * 1024);
    else
      lds_dma16(b_tile + 2 * k0, b_off[i - C::A_INST],
                lds_addr(sB[slot]) + (wave * C::B_INST + i - C::A_INST) * 1024);
  };
  constexpr int NF = C::NRB + C::NCB;         // fragments per k step
  constexpr int NQ = C::NRB * C::NCB;         // MFMAs per k step
  constexpr int NSLOT = NQ / 2;               // MFMA pairs per k step
  constexpr int KS = C::BK / 16;              // 16-deep k steps per stage (2 or 4)
  constexpr int FS = DBL_HEAD_FRAG_SLOTS < NSLOT ? DBL_HEAD_FRAG_SLOTS : NSLOT;
  constexpr int DKS = KS - 1;                 // k steps that carry the stage's DMA
  // MFMA q of a k step multiplies A block q / NCB by B block q % NCB, so fragments are
  // loaded in the order they are first needed: A0, B0 .. B(NCB-1), A1 .. A(NRB-1).
  auto frag_of = [](int f) { return f == 0 ? 0 : (f <= C::NCB ? C::NRB + f - 1 : f - C::NCB); };
  // Slot i of a k step issues MFMA pair i, then the next k step's fragment loads
  // [i NF / FS, (i + 1) NF / FS) (slots i < FS); the stage's DMA instructions are spread
  // evenly over the slots of the first KS - 1 k steps. No load depends on a run-time
  // condition, so the outstanding LDS reads are known at every MFMA and each waits only for
  // its own operands.

  const int nk = d / C::BK;
  // Prologue: stages 0 .. S-2 in flight, stage 0 visible, its first-k-step fragments loaded.
  // (Stages past nk - 1 repeat stage nk - 1 into unused slots.)
#pragma unroll
  for (int j = 0; j < C::S - 1; ++j) {
    const int kj = min(j, nk - 1) * C::BK;
#pragma unroll
    for (int i = 0; i < C::PER_STAGE; ++i) {
      if (j == 0) issue_one(std::integral_constant<int, 0>{}, kj, i);
      if (j == 1) issue_one(std::integral_constant<int, 1 % C::S>{}, kj, i);
      if (j == 2) issue_one(std::integral_constant<int, 2 % C::S>{}, kj, i);
      if (j == 3) issue_one(std::integral_constant<int, 3 % C::S>{}, kj, i);
    }
  }
  wait_vmcnt<(C::S - 2) * C::PER_STAGE>();
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
#pragma unroll
  for (int f = 0; f < NF; ++f) load_frag(0, sA[0], sB[0], 0, frag_of(f));

  // Iteration kt computes stage kt (slot kt % S) in KS k steps; k step s multiplies with
  // fragment set s % 2 while loading set (s + 1) % 2 for k step s + 1. The DMA of stage
  // kt + S - 1 goes to the slot of stage kt - 1 during the first KS - 1 k steps. Before the
  // last k step: wait for stage kt + 1, barrier; the last k step then loads stage kt + 1's
  // first fragments (set 0; after the last stage these read a slot that is never consumed).
  auto body = [&](auto j_c, int kt) {
    constexpr int j = decltype(j_c)::value;
    constexpr int jn = (j + 1) % C::S;            // slot of stage kt + 1
    constexpr int jd = (j + C::S - 1) % C::S;     // slot receiving stage kt + S - 1
    // Stage kt + S - 1 goes to the slot of stage kt - 1, which every wave has finished reading.
    // Past the last stage the copy is repeated from stage nk - 1 into that free slot: the loads
    // stay unconditional, so the outstanding count per wave is always S - 2 stages.
    const int kd = min(kt + C::S - 1, nk - 1) * C::BK;
#pragma unroll
    for (int st = 0; st < KS; ++st) {
      const int cur = st & 1;
      if (st == KS - 1) {
        wait_vmcnt<(C::S - 2) * C::PER_STAGE>();
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
      }
#pragma unroll
      for (int i = 0; i < NSLOT; ++i) {
        mfma(cur, 2 * i);
        mfma(cur, 2 * i + 1);
        if (i < FS) {
#pragma unroll
          for (int f = i * NF / FS; f < (i + 1) * NF / FS; ++f) {
            if (st < KS - 1)
              load_frag(cur ^ 1, sA[j], sB[j], st + 1, frag_of(f));
            else
              load_frag(0, sA[jn], sB[jn], 0, frag_of(f));
          }
        }
        if (st < DKS) {
          constexpr int TS = DKS * NSLOT;
          const int g = st * NSLOT + i;
#pragma unroll
          for (int q = g * C::PER_STAGE / TS; q < (g + 1) * C::PER_STAGE / TS; ++q)
            issue_one(std::integral_constant<int, jd>{}, kd, q);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  int kt0 = 0;
  for (; kt0 + C::S <= nk; kt0 += C::S) {
    body(std::integral_constant<int, 0>{}, kt0);
    body(std::integral_constant<int, 1>{}, kt0 + 1);
    if constexpr (C::S > 2) body(std::integral_constant<int, 2 % C::S>{}, kt0 + 2);
    if constexpr (C::S > 3) body(std::integral_constant<int, 3 % C::S>{}, kt0 + 3);
    if constexpr (C::S > 4) body(std::integral_constant<int, 4 % C::S>{}, kt0 + 4);
  }
  // Remaining nk % S stages.
  if (kt0 < nk) body(std::integral_constant<int, 0>{}, kt0);
  if (kt0 + 1 < nk) body(std::integral_constant<int, 1>{}, kt0 + 1);
  if (C::S > 3 && kt0 + 2 < nk) body(std::integral_constant<int, 2 % C::S>{}, kt0 + 2);
  if (C::S > 4 && kt0 + 3 < nk) body(std::integral_constant<int, 3 % C::S>{}, kt0 + 3);

  wait_vmcnt<0>();

  const int64_t v0w = v0 + wv * kVTile;
  if (v0w >= V) return;
  if constexpr (EPI == kEpiExpand)
    expand_store<C::NRB, C::NCB>(acc, ea, M, V, v0w, m0 + wm * C::TM, lane);
  else
    tile_logsoftmax_store<C::NRB, C::NCB, EPI == kEpiLogSoftmaxArgmax>(
        acc, ea.tls, ea.lmass, ea.amax, M, V, ea.nT, v0w, m0 + wm * C::TM, lane, ea.vec4);
}


// ---------------------------------------------------------------------------------------
// Register-staged kernel (the expander's GEMM, hidden sizes that are a multiple of 64; it was
// the head's main path before the ping-pong kernel): 64-deep stages, so every 128-byte row
// segment of a stage is one request, and a lead of two stages for every load.
// The LDS holds two stages (128 KB); two more stages are in flight in registers (16 16-byte
// loads per thread per stage): during stage kt the threads write stage kt + 1 from registers
// to the LDS slot stage kt - 1 has left and refill those registers with stage kt + 3. The main
// loop needs few VGPRs besides the staging ones (the accumulators are in AGPRs), so the staging
// costs no occupancy. One barrier per stage, before its last k step; the same 128 x 128 wave
// tiles, fragment order and epilogues as the direct-to-LDS kernel.
#ifndef DBL_RS_SPREAD
#define DBL_RS_SPREAD 3
#endif
#ifndef DBL_RS_LSHIFT
#define DBL_RS_LSHIFT 4
#endif
// Tile configuration of the register-staged kernel: BV vocabulary (or output-feature) rows x
// BM branch rows per workgroup, WV x WM waves, each wave 128 x (BM / WM); 64-deep stages.
template <int BV_, int BM_, int WV_, int WM_>
struct RsCfg {
  static constexpr int BV = BV_, BM = BM_, WV = WV_, WM = WM_, BK = 64;
  static constexpr int NW = WV * WM, kThreads = 64 * NW;
  static constexpr int TM = BM / WM, NCB = TM / 32, NRB = 4;
  static constexpr int CPR = BK / 8, ROWB = BK * 2;  // 8 chunks of 16 bytes per 128-byte row
  static constexpr int TILEA = BV * ROWB, TILEB = BM * ROWB;  // bytes per stage and operand
  static constexpr int LDA = BV * CPR / kThreads;    // 16-byte loads per thread, w operand
  static constexpr int LDB = BM * CPR / kThreads;    // 16-byte loads per thread, h operand
  static constexpr int NLD = LDA + LDB;
  static constexpr int KS = BK / 16;                 // k steps per stage (4)
  static constexpr int NQ = NRB * NCB, NSLOT = NQ / 2, NF = NRB + NCB;
  static constexpr int kSpread = DBL_RS_SPREAD;      // k steps carrying the LDS writes
  static constexpr int kShift = DBL_RS_LSHIFT;       // MFMA pairs between a register's write and reload
  static_assert(BV == 128 * WV && kThreads == 256, "waves of 128 vocabulary rows, 256 threads");
  static_assert(LDA >= 1 && LDB >= 1 && BV * CPR % kThreads == 0 && BM * CPR % kThreads == 0,
                "load mapping");
  static_assert(kSpread >= 1 && kSpread <= KS - 1, "staging ends before the stage's barrier");
  static_assert(kShift >= 0 && kShift + kSpread * NSLOT <= KS * NSLOT,
                "every reload issued within the stage");
  static_assert(NF <= 2 * NSLOT, "at most two fragment loads per MFMA pair");
  static_assert(2 * (TILEA + TILEB) <= 160 * 1024, "two stages in LDS");
};
using RsNarrow = RsCfg<128, 256, 1, 4>; // few trunk rows (the expander): 128 x 256 tiles

template <class C, int EPI>
__global__ __launch_bounds__(C::kThreads, 1) void head_bf16_rs_kernel(
    const __bf16* __restrict__ h, const __bf16* __restrict__ w, const EpiArgs ea, int64_t M,
    int64_t V, int d, int n_mtiles) {
  constexpr int BV = C::BV, BM = C::BM, BK = C::BK, WM = C::WM, TM = C::TM, NCB = C::NCB,
                NRB = C::NRB, CPR = C::CPR, ROWB = C::ROWB, LDA = C::LDA, LDB = C::LDB,
                NLD = C::NLD, KS = C::KS, NSLOT = C::NSLOT, NF = C::NF,
                kSpread = C::kSpread, kShift = C::kShift;
  __shared__ __attribute__((aligned(1024))) char sA0[C::TILEA], sB0[C::TILEB], sA1[C::TILEA],
      sB1[C::TILEB];
  char* const sA[2] = {sA0, sA1};
  char* const sB[2] = {sB0, sB1};
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave / WM;
  const int wm = wave % WM;
  int vt, mt;
  tile_of(xcd_remap(blockIdx.x, gridDim.x), gridDim.x / n_mtiles, n_mtiles, &vt, &mt);
  const int64_t v0 = static_cast<int64_t>(vt) * BV;
  const int64_t m0 = static_cast<int64_t>(mt) * BM;

  // Load i of a thread: tile row 32 i + tid / 8, chunk tid % 8 (eight lanes cover a row's 128
  // bytes); stored at chunk c ^ swz(row), swz(row) = (row / 2) % 8, which depends only on
  // tid / 8 here (32 i leaves it unchanged). Rows past V or M are clamped.
  const char* a_tile = reinterpret_cast<const char*>(w + v0 * d);
  const char* b_tile = reinterpret_cast<const char*>(h + m0 * d);
  const int c = tid & 7, r0 = tid >> 3;
  const int lds0 = r0 * ROWB + ((c ^ dma_swz<CPR>(r0)) * 16);
  uint32_t a_off[LDA], b_off[LDB];
#pragma unroll
  for (int i = 0; i < LDA; ++i) {
    const int r = 32 * i + r0;
    const int64_t gv = v0 + r < V ? r : V - 1 - v0;
    a_off[i] = static_cast<uint32_t>(gv * d * 2 + c * 16);
  }
#pragma unroll
  for (int i = 0; i < LDB; ++i) {
    const int r = 32 * i + r0;
    const int64_t gm = m0 + r < M ? r : M - 1 - m0;
    b_off[i] = static_cast<uint32_t>(gm * d * 2 + c * 16);
  }
  u32x4 ra[2][LDA], rb[2][LDB];

  f32x16 acc[NRB][NCB];
#pragma unroll
  for (int rb_ = 0; rb_ < NRB; ++rb_)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[rb_][cb][r] = 0.0f;

  const int tt = 16 * ((lane >> 5) ^ dma_swz<CPR>(lane & 31));
  const int a_base = (wv * kVTile + (lane & 31)) * ROWB;
  const int b_base = (wm * TM + (lane & 31)) * ROWB;
  bf16x8 af[2][NRB], bfr[2][NCB];
  auto load_frag = [&](int set, const char* As, const char* Bs, int ks, int i) {
    const int x = (32 * ks) ^ tt;
    if (i < NRB)
      af[set][i] = *reinterpret_cast<const bf16x8*>(As + a_base + i * 32 * ROWB + x);
    else
      bfr[set][i - NRB] = *reinterpret_cast<const bf16x8*>(Bs + b_base + (i - NRB) * 32 * ROWB + x);
  };
  auto mfma = [&](int set, int q) {
    const int rb_ = q / NCB, cb = q % NCB;
    acc[rb_][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[set][rb_], bfr[set][cb],
                                                            acc[rb_][cb], 0, 0, 0);
  };
  const int nk = d / BK;
  // global -> registers (stage s, clamped to the last stage) and registers -> LDS, one 16-byte
  // load of one operand at a time (q < LDA: w, else h)
  // Stages past the last (the pipeline's final three reloads) read the tile's first 16 bytes in
  // every lane: one cached request instead of a stage of operand traffic; never consumed.
  auto gload = [&](auto buf_c, int s, int q) {
    constexpr int buf = decltype(buf_c)::value;
    const bool live = s < nk;
    if (q < LDA)
      ra[buf][q] = *reinterpret_cast<const u32x4*>(a_tile + (live ? a_off[q] + s * ROWB : 0u));
    else
      rb[buf][q - LDA] =
          *reinterpret_cast<const u32x4*>(b_tile + (live ? b_off[q - LDA] + s * ROWB : 0u));
  };
  auto swrite = [&](auto buf_c, auto slot_c, int q) {
    constexpr int buf = decltype(buf_c)::value, slot = decltype(slot_c)::value;
    if (q < LDA)
      *reinterpret_cast<u32x4*>(sA[slot] + lds0 + q * 32 * ROWB) = ra[buf][q];
    else
      *reinterpret_cast<u32x4*>(sB[slot] + lds0 + (q - LDA) * 32 * ROWB) = rb[buf][q - LDA];
  };
  auto frag_of = [](int f) { return f == 0 ? 0 : (f <= NCB ? NRB + f - 1 : f - NCB); };

  // Prologue: stage 0 in LDS slot 0, stage 1 in registers (buffer 1), stage 2 in flight
  // (buffer 0), stage 0's first fragments loaded.
#pragma unroll
  for (int q = 0; q < NLD; ++q) gload(std::integral_constant<int, 0>{}, 0, q);
#pragma unroll
  for (int q = 0; q < NLD; ++q) gload(std::integral_constant<int, 1>{}, 1, q);
#pragma unroll
  for (int q = 0; q < NLD; ++q) {
    swrite(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{}, q);
    gload(std::integral_constant<int, 0>{}, 2, q);
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
#pragma unroll
  for (int f = 0; f < NF; ++f) load_frag(0, sA[0], sB[0], 0, frag_of(f));

  // Stage kt (slot j = kt % 2): its first kSpread k steps write stage kt + 1 (registers j ^ 1)
  // to slot j ^ 1, and each of those registers is reloaded with stage kt + 3 kShift MFMA pairs
  // after its write; registers j hold stage kt + 2. Before the last k step: LDS writes done,
  // barrier; the last k step loads stage kt + 1's first fragments.
  auto body = [&](auto j_c, int kt) {
    constexpr int j = decltype(j_c)::value;
    constexpr int jn = j ^ 1;
#pragma unroll
    for (int st = 0; st < KS; ++st) {
      const int cur = st & 1;
      if (st == KS - 1) {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
      }
#pragma unroll
      for (int i = 0; i < NSLOT; ++i) {
        mfma(cur, 2 * i);
        mfma(cur, 2 * i + 1);
        // Fragments i NF / NSLOT .. (i + 1) NF / NSLOT - 1 of the next k step (in the order
        // the MFMAs consume them).
#pragma unroll
        for (int f = i * NF / NSLOT; f < (i + 1) * NF / NSLOT; ++f) {
          if (st < KS - 1)
            load_frag(cur ^ 1, sA[j], sB[j], st + 1, frag_of(f));
          else
            load_frag(0, sA[jn], sB[jn], 0, frag_of(f));
        }
        {
          // Register q is written to LDS at slot q TS / NLD of the first kSpread k steps and
          // reloaded kShift slots later.
          constexpr int TS = kSpread * NSLOT;
          const int g = st * NSLOT + i;
          if (st < kSpread) {
#pragma unroll
            for (int q = g * NLD / TS; q < (g + 1) * NLD / TS; ++q)
              swrite(std::integral_constant<int, jn>{}, std::integral_constant<int, jn>{}, q);
          }
          const int gl = g - kShift;
          if (gl >= 0 && gl < TS) {
#pragma unroll
            for (int q = gl * NLD / TS; q < (gl + 1) * NLD / TS; ++q)
              gload(std::integral_constant<int, jn>{}, kt + 3, q);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  int kt0 = 0;
  for (; kt0 + 2 <= nk; kt0 += 2) {
    body(std::integral_constant<int, 0>{}, kt0);
    body(std::integral_constant<int, 1>{}, kt0 + 1);
  }
  if (kt0 < nk) body(std::integral_constant<int, 0>{}, kt0);
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");

  // Keep the accumulators in AGPRs past the loop's exit (otherwise all of them are copied to
  // VGPRs right here, leaving the epilogue no registers to work in).
#pragma unroll
  for (int rb_ = 0; rb_ < NRB; ++rb_)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) asm volatile("" : "+a"(acc[rb_][cb]));

  const int64_t v0w = v0 + wv * kVTile;
  if (v0w >= V) return;
  if constexpr (EPI == kEpiExpand) {
    expand_store<NRB, NCB>(acc, ea, M, V, v0w, m0 + wm * TM, lane);
  } else if constexpr (DBL_HEAD_XP) {
    // The last stage's slot is free once every wave has passed that stage's barrier (its reads
    // came before it; the last k step reads the other slot): 16 KB of it per wave for the
    // stores.
    static_assert(C::NW == 4 && C::TILEA / 2 >= 32 * 512 && C::TILEB / 2 >= 32 * 512,
                  "16 KB of LDS per wave for the transposed stores");
    const int jl = (nk - 1) & 1;
    char* const xp = (jl ? (wave < 2 ? sA1 : sB1) : (wave < 2 ? sA0 : sB0)) +
                     (wave & 1) * (wave < 2 ? C::TILEA / 2 : C::TILEB / 2);
    tile_logsoftmax_store_lds<NRB, NCB, EPI == kEpiLogSoftmaxArgmax>(
        acc, ea.tls, ea.lmass, ea.amax, M, V, ea.nT, v0w, m0 + wm * TM, lane, ea.vec4, xp);
  } else
    tile_logsoftmax_store<NRB, NCB, EPI == kEpiLogSoftmaxArgmax>(
        acc, ea.tls, ea.lmass, ea.amax, M, V, ea.nT, v0w, m0 + wm * TM, lane, ea.vec4);
}

// ---------------------------------------------------------------------------------------
// Ping-pong variant (the head for hidden sizes that are a multiple of 64): 8 waves, two per
// SIMD (the dispatcher places waves w and w + 4 of a workgroup on the same SIMD, waves 0-3 on
// four different ones), in two groups of four that take turns between workgroup barriers: one
// group issues MFMAs on fragments already in its registers while the other reads its next
// fragments from LDS and issues global -> LDS copies, so the MFMA-issuing wave never waits on
// memory and each SIMD's matrix pipe is fed by one wave or the other.
//   * Workgroup tile 256 vocabulary x 256 branch rows, 64-deep stages; each wave owns a 128 x 64
//     output block (one vocabulary tile for 64 branch rows). A turn covers 32 of a stage's 64 k:
//     12 fragment reads, 16 MFMAs.
//   * LDS (160 KB): three slots for the w rows of a stage (stage s in slot s % 3) and two for
//     the h rows (slot s % 2), filled by global_load_lds_dwordx4. Every memory half of every
//     turn issues the same 16 KB of copies (4 instructions per wave; each group copies half of
//     each operand's rows): even turn 2 s the h rows of stage s + 1, odd turn 2 s + 1 the w rows
//     of stage s + 2, so w (streamed from HBM) has two stages of lead and h (re-read from L2)
//     one. Copies issued in one burst per stage stretched the memory halves and cost 6%.
struct PpCfg {
  static constexpr int BV = 256, BM = 256, BK = 64, kThreads = 512;
  static constexpr int TM = 64, NRB = 4, NCB = 2;  // wave block: 128 ids x 64 branch rows
  static constexpr int ROWB = 128;                 // bytes per LDS row (64 bf16)
  static constexpr int TILE = 256 * ROWB;          // bytes per operand per stage (32 KB)
  static_assert(5 * TILE <= 160 * 1024 && 8 * 32 * 512 <= 5 * TILE, "LDS budget");
};

__device__ __forceinline__ void pp_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

template <bool ARG>
__global__ __launch_bounds__(512, 1) void head_bf16_pp_kernel(
    const __bf16* __restrict__ h, const __bf16* __restrict__ w, const EpiArgs ea, int64_t M,
    int64_t V, int d, int n_mtiles) {
  using C = PpCfg;
  constexpr int ROWB = C::ROWB, TILE = C::TILE, NRB = C::NRB, NCB = C::NCB;
  constexpr int BOFF = 3 * TILE;  // the two h slots follow the three w slots
  // After the loop the first 128 KB hold the epilogue's per-wave 16 KB store staging.
  __shared__ __attribute__((aligned(1024))) char smem[5 * TILE];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;  // group 0 computes first in every pair of turns
  const int wv = wave & 1;    // vocabulary half of the workgroup tile
  const int wm = wave >> 1;   // branch-row quarter (0, 1 in group 0; 2, 3 in group 1)
  const int q = wave & 3;
  int vt, mt;
  tile_of(xcd_remap(blockIdx.x, gridDim.x), gridDim.x / n_mtiles, n_mtiles, &vt, &mt);
  const int64_t v0 = static_cast<int64_t>(vt) * C::BV;
  const int64_t m0 = static_cast<int64_t>(mt) * C::BM;

  // Copies: wave q of group g copies rows 128 g + (4 q + i) * 8 + lane / 8 (i < 4) of the w tile
  // and of the h tile; lane % 8 is its 16-byte chunk's place in the LDS row and it fetches
  // chunk (lane % 8) ^ swz(row) of that row (rows past V or M repeat the last one). A scalar
  // tile base plus 32-bit lane offsets (at most 512 d bytes).
  const char* srcA = reinterpret_cast<const char*>(w + v0 * d);
  const char* srcB = reinterpret_cast<const char*>(h + m0 * d);
  uint32_t offA[4], offB[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 128 * grp + (4 * q + i) * 8 + lane / 8;
    const int c = (lane % 8) ^ dma_swz<8>(r);
    const int64_t ga = r < V - v0 ? r : V - v0 - 1;
    const int64_t gb = r < M - m0 ? r : M - m0 - 1;
    offA[i] = static_cast<uint32_t>(ga * d * 2 + c * 16);
    offB[i] = static_cast<uint32_t>(gb * d * 2 + c * 16);
  }
  const uint32_t lds_row = lds_addr(smem) + (16 * grp + 4 * q) * 1024;
  auto copy_A = [&](int s, int slot) {
    const char* base = srcA + static_cast<int64_t>(s) * (2 * C::BK);
#pragma unroll
    for (int i = 0; i < 4; ++i) lds_dma16(base, offA[i], lds_row + slot * TILE + i * 1024);
  };
  auto copy_B = [&](int s, int slot) {
    const char* base = srcB + static_cast<int64_t>(s) * (2 * C::BK);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      lds_dma16(base, offB[i], lds_row + BOFF + slot * TILE + i * 1024);
  };

  f32x16 acc[NRB][NCB];
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[rb][cb][r] = 0.0f;

  // Fragments of a turn: lane l reads row l % 32 of each 32-row block, 8 k values from
  // 8 (l / 32) of each 16-wide k step (chunk 2 kk + l / 32, stored at chunk ^ swz(row)).
  const int tt = 16 * ((lane >> 5) ^ dma_swz<8>(lane & 31));
  const int a_base = (wv * kVTile + (lane & 31)) * ROWB;
  const int b_base = BOFF + (wm * C::TM + (lane & 31)) * ROWB;
  bf16x8 af[2][NRB], bfr[2][NCB];
  auto load_frags = [&](int aslot, int bslot, int kk0) {
    const char* sa = smem + aslot * TILE;
    const char* sb = smem + bslot * TILE;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int x = (32 * (kk0 + ks)) ^ tt;
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
        af[ks][rb] = *reinterpret_cast<const bf16x8*>(sa + a_base + rb * 32 * ROWB + x);
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
        bfr[ks][cb] = *reinterpret_cast<const bf16x8*>(sb + b_base + cb * 32 * ROWB + x);
    }
  };
  auto compute = [&]() {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[ks][rb], bfr[ks][cb],
                                                                 acc[rb][cb], 0, 0, 0);
  };

  const int nk = d / C::BK;
  const int H = 2 * nk;  // turns per group
  // Turn t of a group: its memory half (fragments of k half t % 2 of stage s = t / 2, plus the
  // turn's copies into slots that stage s - 1 has left), a barrier, its compute half, a barrier.
  // Group 1 runs one barrier behind group 0, so each half of one group coincides with the other
  // half of the other. At odd turns every wave waits for its own copies of stage s + 1 (all but
  // the 4 instructions of stage s + 2 just issued) before the barrier that opens the first
  // memory half reading stage s + 1; a slot is refilled only after the barrier that closes the
  // last memory half reading it.
  auto turn = [&](int t, int a3, int b2) {  // a3 = (t / 2) % 3, b2 = (t / 2) % 2
    const int s = t >> 1;
    load_frags(a3, b2, (t & 1) * 2);
    if (!(t & 1)) {
      if (t >= 2 && s + 1 < nk) copy_B(s + 1, b2 ^ 1);
    } else {
      if (s + 2 < nk) copy_A(s + 2, a3 == 0 ? 2 : a3 - 1);
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if ((t & 1) && grp == 1) {
      if (s + 2 < nk) wait_vmcnt<4>(); else wait_vmcnt<0>();
    }
    pp_barrier();
    compute();
    if ((t & 1) && grp == 0) {
      if (s + 2 < nk) wait_vmcnt<4>(); else wait_vmcnt<0>();
    }
    if (!(grp == 1 && t == H - 1)) pp_barrier();
  };
  copy_A(0, 0);
  copy_B(0, 0);
  if (nk > 1) {
    copy_A(1, 1);
    copy_B(1, 1);
    wait_vmcnt<8>();
  } else {
    wait_vmcnt<0>();
  }
  pp_barrier();
  if (grp == 1) pp_barrier();
  int a3 = 0;
  for (int t = 0; t < H; t += 2) {
    turn(t, a3, (t >> 1) & 1);
    turn(t + 1, a3, (t >> 1) & 1);
    a3 = a3 == 2 ? 0 : a3 + 1;
  }

#pragma unroll
  for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) asm volatile("" : "+a"(acc[rb][cb]));

  // No memory half reads the slots any more (group 0 passed the barrier closing the last one;
  // group 1 reads none in its last compute half) and every copy has landed, so each wave stages
  // its stores in its own 16 KB of them.
  const int64_t v0w = v0 + wv * kVTile;
  if (v0w >= V) return;
  tile_logsoftmax_store_lds<NRB, NCB, ARG>(acc, ea.tls, ea.lmass, ea.amax, M, V, ea.nT, v0w,
                                           m0 + wm * C::TM, lane, ea.vec4, smem + wave * 16384);
}

// fp32 path: workgroup (vocabulary tile t, 4 branch rows); thread j owns id 128 t + j.
constexpr int kF32Rows = 4;
constexpr int kF32DChunk = 512;

__global__ __launch_bounds__(128) void head_f32_kernel(const float* __restrict__ h,
                                                       const float* __restrict__ w,
                                                       float* __restrict__ tls,
                                                       float* __restrict__ lmass,
                                                       uint64_t* __restrict__ amax, int64_t M,
                                                       int64_t V, int d, int nT) {
  __shared__ float hs[kF32Rows][kF32DChunk];
  __shared__ float red[2][kF32Rows];
  __shared__ int redi[2][kF32Rows];
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
    if (amax) {  // first id of the tile holding the maximum
      int first = valid && acc[r] == mx ? j : kVTile;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) first = min(first, __shfl_xor(first, o));
      if ((j & 63) == 0) redi[wave][r] = first;
      __syncthreads();
      first = min(redi[0][r], redi[1][r]);
      const int64_t m = m0 + r;
      if (j == 0 && m < M && first < kVTile)
        atomicMax(reinterpret_cast<unsigned long long*>(amax + m),
                  static_cast<unsigned long long>(argmax_key(mx, static_cast<int64_t>(t) * kVTile + first)));
      __syncthreads();
    }
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

// Clears the per-row argmax keys before the head kernel accumulates into them.
__global__ __launch_bounds__(256) void zero_u64_kernel(uint64_t* __restrict__ p, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = 0;
}

constexpr int kLseRegs = 32;

// lse[m] = log sum_t exp(lmass[m, t]); one wave per row. With argmax requested, also decodes
// the row's winning key into the vocabulary id.
__global__ __launch_bounds__(256) void lse_finalize_kernel(const float* __restrict__ lmass,
                                                           float* __restrict__ lse,
                                                           const uint64_t* __restrict__ amax,
                                                           int32_t* __restrict__ argmax,
                                                           int64_t M, int nT) {
  const int64_t m = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (m >= M) return;
  const float* row = lmass + m * nT;
  // The maximum, then the sum of exponentials relative to it, each lane over ids lane, lane +
  // 64, ... in that order. Rows of up to 64 kLseRegs tiles (V <= 262,144) are loaded once, all
  // loads issued together, and kept in registers for both passes; longer rows are read twice.
  float mx = -INFINITY, s = 0.0f;
  if (nT <= 64 * kLseRegs) {
    float x[kLseRegs];
#pragma unroll
    for (int i = 0; i < kLseRegs; ++i) {
      const int t = lane + 64 * i;
      x[i] = t < nT ? row[t] : -INFINITY;
    }
#pragma unroll
    for (int i = 0; i < kLseRegs; ++i) mx = fmaxf(mx, x[i]);
    const float gmx = wave_max(mx);
    if (gmx > -INFINITY) {
#pragma unroll
      for (int i = 0; i < kLseRegs; ++i)
        if (lane + 64 * i < nT) s += x[i] > -INFINITY ? __expf(x[i] - gmx) : 0.0f;
    }
    mx = gmx;
  } else {
#pragma unroll 4
    for (int t = lane; t < nT; t += 64) mx = fmaxf(mx, row[t]);
    const float gmx = wave_max(mx);
    if (gmx > -INFINITY) {
#pragma unroll 4
      for (int t = lane; t < nT; t += 64) {
        const float x = row[t];
        s += x > -INFINITY ? __expf(x - gmx) : 0.0f;
      }
    }
    mx = gmx;
  }
  const float gmx = mx;
  s = wave_sum(s);
  if (lane == 0) {
    lse[m] = gmx + __logf(s);
    if (argmax) {
      const uint64_t key = amax[m];
      argmax[m] = key ? static_cast<int32_t>(0xFFFFFFFFu - static_cast<uint32_t>(key)) : -1;
    }
  }
}

}  // namespace

hipError_t launch_head(const HeadArgs& a, hipStream_t stream) {
  const int nT = static_cast<int>((a.V + kVTile - 1) / kVTile);
  uint64_t* amax = a.argmax ? a.amax_keys : nullptr;
  if (amax) {
    const int64_t zb = (a.M + 255) / 256;
    if (zb > 0x7fffffff) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(zero_u64_kernel, dim3(static_cast<unsigned>(zb)), dim3(256), 0, stream,
                       amax, a.M);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.dtype_bf16) {
    const int n_mtiles = static_cast<int>((a.M + Cfg::BM - 1) / Cfg::BM);
    const int64_t n_vtiles = (a.V + Cfg::BV - 1) / Cfg::BV;
    const int64_t nwg = n_vtiles * n_mtiles;
    if (nwg > 0x7fffffff) return hipErrorInvalidConfiguration;
    const int vec4 = (a.V % 4 == 0) ? 1 : 0;
    const __bf16* h = static_cast<const __bf16*>(a.h);
    const __bf16* w = static_cast<const __bf16*>(a.w);
    if (a.d % PpCfg::BK == 0) {
      const int dm = static_cast<int>((a.M + PpCfg::BM - 1) / PpCfg::BM);
      const int64_t dwg = ((a.V + PpCfg::BV - 1) / PpCfg::BV) * dm;
      if (dwg > 0x7fffffff) return hipErrorInvalidConfiguration;
      EpiArgs ea{};
      ea.tls = a.tls;
      ea.lmass = a.lmass;
      ea.amax = amax;
      ea.nT = nT;
      ea.vec4 = vec4;
      const dim3 grid(static_cast<unsigned>(dwg)), block(PpCfg::kThreads);
      if (amax)
        hipLaunchKernelGGL(head_bf16_pp_kernel<true>, grid, block, 0, stream, h, w, ea, a.M, a.V,
                           a.d, dm);
      else
        hipLaunchKernelGGL(head_bf16_pp_kernel<false>, grid, block, 0, stream, h, w, ea, a.M,
                           a.V, a.d, dm);
    } else if (a.d % DCfg::BK == 0) {
      const int dm = static_cast<int>((a.M + DCfg::BM - 1) / DCfg::BM);
      const int64_t dwg = ((a.V + DCfg::BV - 1) / DCfg::BV) * dm;
      if (dwg > 0x7fffffff) return hipErrorInvalidConfiguration;
      const dim3 grid(static_cast<unsigned>(dwg)), block(DCfg::kThreads);
      EpiArgs ea{};
      ea.tls = a.tls;
      ea.lmass = a.lmass;
      ea.amax = amax;
      ea.nT = nT;
      ea.vec4 = vec4;
      if (amax)
        hipLaunchKernelGGL((head_bf16_dma_kernel<DCfg, kEpiLogSoftmaxArgmax>), grid, block, 0,
                           stream, h, w, ea, a.M, a.V, a.d, dm);
      else
        hipLaunchKernelGGL((head_bf16_dma_kernel<DCfg, kEpiLogSoftmax>), grid, block, 0, stream,
                           h, w, ea, a.M, a.V, a.d, dm);
    } else {
      const dim3 grid(static_cast<unsigned>(nwg)), block(Cfg::kThreads);
      if (amax)
        hipLaunchKernelGGL((head_bf16_kernel<Cfg, true>), grid, block, 0, stream, h, w, a.tls,
                           a.lmass, amax, a.M, a.V, a.d, nT, n_mtiles, vec4);
      else
        hipLaunchKernelGGL((head_bf16_kernel<Cfg, false>), grid, block, 0, stream, h, w, a.tls,
                           a.lmass, amax, a.M, a.V, a.d, nT, n_mtiles, vec4);
    }
  } else {
    const int64_t mblocks = (a.M + kF32Rows - 1) / kF32Rows;
    if (mblocks > 65535) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(head_f32_kernel, dim3(nT, static_cast<unsigned>(mblocks)), dim3(128), 0,
                       stream, static_cast<const float*>(a.h), static_cast<const float*>(a.w),
                       a.tls, a.lmass, amax, a.M, a.V, a.d, nT);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t lse_blocks = (a.M + 3) / 4;
  hipLaunchKernelGGL(lse_finalize_kernel, dim3(static_cast<unsigned>(lse_blocks)), dim3(256), 0,
                     stream, a.lmass, a.lse, amax, amax ? a.argmax : nullptr, a.M, nT);
  return hipGetLastError();
}

namespace {

// Category-prior head: l[b, z] = sum_j U[z, j] h_anchor[b, j] + e[z] in fp32 accumulation.
// One workgroup per block; every category's dot product is a workgroup reduction.
__global__ __launch_bounds__(256) void prior_head_kernel(const __bf16* __restrict__ ha,
                                                         const __bf16* __restrict__ U,
                                                         const __bf16* __restrict__ e,
                                                         float* __restrict__ ell, int R, int d) {
  __shared__ float red[4];
  const int64_t b = blockIdx.x;
  const __bf16* hb = ha + b * d;
  for (int z = 0; z < R; ++z) {
    const __bf16* u = U + static_cast<int64_t>(z) * d;
    float s = 0.0f;
    for (int j = threadIdx.x; j < d; j += 256)
      s = fmaf(static_cast<float>(u[j]), static_cast<float>(hb[j]), s);
    s = wave_sum(s);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) ell[b * R + z] = ((red[0] + red[1]) + (red[2] + red[3])) + static_cast<float>(e[z]);
    __syncthreads();
  }
}

}  // namespace

// Expander GEMMs have few trunk rows (B*K) and a wide output (R*d): when 256-row tiles would not
// give every CU a workgroup, 128-row tiles double the workgroup count (the weight slab each
// pair of them shares is read from L2).
using ECfg = DmaCfg<32, 4, 128, 2>;
constexpr int kCus = 256;

template <class C>
hipError_t launch_expand_cfg(const ExpandArgs& a, int64_t N, hipStream_t stream) {
  const int dm = static_cast<int>((a.M + C::BM - 1) / C::BM);
  const int64_t dwg = ((N + C::BV - 1) / C::BV) * dm;
  if (dwg > 0x7fffffff || a.d % C::BK != 0) return hipErrorInvalidConfiguration;
  EpiArgs ea{};
  ea.out = static_cast<__bf16*>(a.out);
  ea.bias = static_cast<const __bf16*>(a.c);
  ea.hres = static_cast<const __bf16*>(a.h);
  ea.dres = a.d;
  hipLaunchKernelGGL((head_bf16_dma_kernel<C, kEpiExpand>), dim3(static_cast<unsigned>(dwg)),
                     dim3(C::kThreads), 0, stream, static_cast<const __bf16*>(a.h),
                     static_cast<const __bf16*>(a.W), ea, a.M, N, a.d, dm);
  return hipGetLastError();
}

// Register-staged expander for few trunk rows: 128 output features x 256 rows per workgroup, so
// every weight row is streamed once and the grid still covers the chip.
template <class C>
hipError_t launch_expand_rs(const ExpandArgs& a, int64_t N, hipStream_t stream) {
  const int dm = static_cast<int>((a.M + C::BM - 1) / C::BM);
  const int64_t dwg = ((N + C::BV - 1) / C::BV) * dm;
  if (dwg > 0x7fffffff || a.d % C::BK != 0) return hipErrorInvalidConfiguration;
  EpiArgs ea{};
  ea.out = static_cast<__bf16*>(a.out);
  ea.bias = static_cast<const __bf16*>(a.c);
  ea.hres = static_cast<const __bf16*>(a.h);
  ea.dres = a.d;
  hipLaunchKernelGGL((head_bf16_rs_kernel<C, kEpiExpand>), dim3(static_cast<unsigned>(dwg)),
                     dim3(C::kThreads), 0, stream, static_cast<const __bf16*>(a.h),
                     static_cast<const __bf16*>(a.W), ea, a.M, N, a.d, dm);
  return hipGetLastError();
}
hipError_t launch_expand(const ExpandArgs& a, hipStream_t stream) {
  const int64_t N = a.R * a.d;
  const int64_t wg256 = ((N + DCfg::BV - 1) / DCfg::BV) * ((a.M + DCfg::BM - 1) / DCfg::BM);
  if (wg256 < kCus) {
    if (a.d % RsNarrow::BK == 0) return launch_expand_rs<RsNarrow>(a, N, stream);
    return launch_expand_cfg<ECfg>(a, N, stream);
  }
  return launch_expand_cfg<DCfg>(a, N, stream);
}

hipError_t launch_prior_head(const PriorHeadArgs& a, hipStream_t stream) {
  if (a.B > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(prior_head_kernel, dim3(static_cast<unsigned>(a.B)), dim3(256), 0, stream,
                     static_cast<const __bf16*>(a.h_anchor), static_cast<const __bf16*>(a.U),
                     static_cast<const __bf16*>(a.e), a.ell, a.R, a.d);
  return hipGetLastError();
}

}  // namespace dbl
