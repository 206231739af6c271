// Wavefront (64-lane) helpers shared by the sampler and verifier kernels. Internal.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "contract.hpp"
#include "kernels.hpp"

namespace dbl {

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// 16-byte load of data that a launch reads exactly once (the rows of the acceptance-mass stream,
// a target row), with the non-temporal hint so that it does not displace cached lines: a linear
// 1.4 GB read measured 7.0-7.2 TB/s this way against 6.2-6.5 TB/s with plain loads, the
// verification stream 6-9% faster and the expected-length stream 11% faster.
#ifndef DBL_NT_LOADS
#define DBL_NT_LOADS 1
#endif
typedef float stream_f32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 load_stream4(const float* p) {
#if DBL_NT_LOADS
  const stream_f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const stream_f32x4*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
#else
  return *reinterpret_cast<const float4*>(p);
#endif
}

// Value of lane l (wave-uniform l) in every lane: v_readlane on each 32-bit half, a few cycles
// instead of an LDS-crossbar shuffle.
__device__ __forceinline__ uint64_t lane_u64(uint64_t v, int l) {
  const uint32_t lo = static_cast<uint32_t>(
      __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(v)), l));
  const uint32_t hi = static_cast<uint32_t>(
      __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(v >> 32)), l));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}
__device__ __forceinline__ double lane_f64(double v, int l) {
  return __longlong_as_double(
      static_cast<long long>(lane_u64(static_cast<uint64_t>(__double_as_longlong(v)), l)));
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ double wave_max_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
  return v;
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Inclusive prefix sum over the 64 lanes.
__device__ __forceinline__ uint64_t wave_incl_scan_u64(uint64_t v) {
  const int lane = lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t t = __shfl_up(v, o);
    if (lane >= o) v += t;
  }
  return v;
}

// Unnormalised log prior of category z = lane (lanes >= R hold -inf) from raw = l_lane (any
// value on lanes >= R): l_z / Z_T, or for Z_T = 0, 0 at the lowest-index maximum of l and -inf
// elsewhere.
__device__ __forceinline__ double prior_log_weight_of(float raw, int R, float z_temp) {
  const int lane = lane_id();
  const float l = lane < R ? raw : -INFINITY;
  if (z_temp > 0.0f)
    return lane < R ? static_cast<double>(l) / static_cast<double>(z_temp) : -INFINITY;
  float mx = l;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  const uint64_t hit = __ballot(lane < R && l == mx);
  const int top = __ffsll(static_cast<unsigned long long>(hit)) - 1;
  return lane == top ? 0.0 : -INFINITY;
}

// The same, loading l from the block's prior row (clamped index: every lane's load is in bounds).
__device__ __forceinline__ double prior_log_weight(const float* prior_row, int R, float z_temp) {
  return prior_log_weight_of(prior_row[min(lane_id(), R - 1)], R, z_temp);
}

// w_z = exp(L_z - max L) / sum_z exp(L_z - max L), the sum taken over ascending z with each
// addition rounded separately; every lane computes the identical sum. An all -inf row (an
// impossible prefix) gives all-zero weights.
__device__ __forceinline__ double normalize_weight(double L, int R) {
  double mx = lane_f64(L, 0);
  for (int z = 1; z < R; ++z) mx = fmax(mx, lane_f64(L, z));
  if (!(mx > -INFINITY)) return 0.0;
  const double e = dexp64(__dsub_rn(L, mx));
  double S = 0.0;
  for (int z = 0; z < R; ++z) S = __dadd_rn(S, lane_f64(e, z));
  return e / S;
}

// normalize_weight for several positions per wavefront: lanes in segments of G (a power of two,
// R <= G <= 64), lane z of a segment holding category z's log weight. Each segment gets exactly
// what normalize_weight gives a wavefront holding the same values (same operations, same order).
// Up to 16 lanes per segment the segment's values are gathered with all shuffles in flight
// before the ordered maximum and sum (fixed-count loops); wider segments walk them in turn.
template <int G>
__device__ __forceinline__ double normalize_weight_seg(double L, int R) {
  const int base = lane_id() & ~(G - 1);
  if constexpr (G <= 16) {
    double v[G];
#pragma unroll
    for (int z = 0; z < G; ++z) v[z] = __shfl(L, base + z);
    double mx = v[0];
#pragma unroll
    for (int z = 1; z < G; ++z)
      if (z < R) mx = fmax(mx, v[z]);
    if (!(mx > -INFINITY)) return 0.0;
    const double e = dexp64(__dsub_rn(L, mx));
#pragma unroll
    for (int z = 0; z < G; ++z) v[z] = __shfl(e, base + z);
    double S = 0.0;
#pragma unroll
    for (int z = 0; z < G; ++z)
      if (z < R) S = __dadd_rn(S, v[z]);
    return e / S;
  } else {
    double mx = __shfl(L, base);
    for (int z = 1; z < R; ++z) mx = fmax(mx, __shfl(L, base + z));
    if (!(mx > -INFINITY)) return 0.0;
    const double e = dexp64(__dsub_rn(L, mx));
    double S = 0.0;
    for (int z = 0; z < R; ++z) S = __dadd_rn(S, __shfl(e, base + z));
    return e / S;
  }
}

// The category z ~ q_{Z_T} of block b by inverse CDF on floor(w_z 2^40); all lanes agree.
__device__ __forceinline__ int draw_category(const BlockArgs& a, int64_t b) {
  const int lane = lane_id();
  const int R = static_cast<int>(a.R);
  const double w = normalize_weight(prior_log_weight(a.prior + b * a.R, R, a.z_temp), R);
  const uint64_t qz = lane < R ? quant40d(w) : 0;
  uint64_t Z = 0;
  for (int z = 0; z < R; ++z) Z += lane_u64(qz, z);
  if (Z == 0) return -1;
  const uint32_t r = draw(a.seed, kCategory, 0, static_cast<uint64_t>(a.seq_offset + b), a.step);
  const uint64_t T = icdf_threshold(r, Z);
  uint64_t cum = 0;
  for (int z = 0; z < R; ++z) {
    cum += lane_u64(qz, z);
    if (cum > T) return z;
  }
  return R - 1;  // unreachable: cum reaches Z > T
}

// Workgroup inverse CDF over n integer weights weigh(load(i)), i < n (every thread of a
// 256-thread workgroup calls it, with the same n and r): each thread sums a contiguous run, a
// workgroup scan gives the total Z and the run holding T = floor(r Z / 2^32), and that run's
// thread finds the smallest index whose inclusive cumulative weight exceeds T. Runs of up to
// kRunRegs values (n <= 2048) are loaded into registers first, all with in-bounds (clamped)
// indices, and weighed afterwards, so the loads are in flight together (a weight function with
// branches would otherwise wait for each load in turn); longer runs are walked twice. Returns
// the index (-1 when Z = 0) with T and the cumulative weight before it. `lds` must hold 8
// uint64.
struct Pick {
  int i;
  uint64_t T, before;
};
constexpr int kRunRegs = 8;

template <class LoadFn, class WeighFn>
__device__ Pick pick_block(int n, LoadFn load, WeighFn weigh, uint32_t r, uint64_t* lds) {
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  if (n <= 0) return Pick{-1, 0, 0};
  const int per = (n + 255) / 256;
  const int i0 = min(n, tid * per), i1 = min(n, i0 + per);
  const bool regs = per <= kRunRegs;  // workgroup-uniform
  uint64_t wr[kRunRegs];
  uint64_t part = 0;
  if (regs) {
    const int last = (i1 > i0 ? i1 : n) - 1;  // a valid index for the clamped loads
    decltype(load(0)) raw[kRunRegs];
#pragma unroll
    for (int j = 0; j < kRunRegs; ++j) raw[j] = load(min(i0 + j, last));
#pragma unroll
    for (int j = 0; j < kRunRegs; ++j) {
      wr[j] = i0 + j < i1 ? static_cast<uint64_t>(weigh(raw[j])) : 0;
      part += wr[j];
    }
  } else {
    for (int i = i0; i < i1; ++i) part += weigh(load(i));
  }
  uint64_t incl = wave_incl_scan_u64(part);
  if (lane == 63) lds[wave] = incl;
  __syncthreads();
  uint64_t base = 0, Z = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (w < wave) base += lds[w];
    Z += lds[w];
  }
  __syncthreads();
  if (Z == 0) return Pick{-1, 0, 0};
  const uint64_t T = icdf_threshold(r, Z);
  incl += base;
  const uint64_t excl = incl - part;
  if (excl <= T && T < incl) {  // exactly one thread's run holds the threshold
    uint64_t c = excl;
    if (regs) {
      int found = -1;
      uint64_t cb = 0;
#pragma unroll
      for (int j = 0; j < kRunRegs; ++j) {
        if (found < 0 && c + wr[j] > T) {  // the run's total exceeds T: the first hit is in it
          found = i0 + j;
          cb = c;
        }
        c += wr[j];
      }
      lds[4] = static_cast<uint64_t>(found);
      lds[5] = cb;
    } else {
      for (int i = i0; i < i1; ++i) {
        const uint64_t wi = weigh(load(i));
        if (c + wi > T) {
          lds[4] = static_cast<uint64_t>(i);
          lds[5] = c;
          break;
        }
        c += wi;
      }
    }
  }
  __syncthreads();
  const Pick pk{static_cast<int>(lds[4]), T, lds[5]};
  __syncthreads();
  return pk;
}

// The selection of pick_block, index only.
template <class LoadFn, class WeighFn>
__device__ int select_block(int n, LoadFn load, WeighFn weigh, uint32_t r, uint64_t* lds) {
  return pick_block(n, load, weigh, r, lds).i;
}

__device__ __forceinline__ uint64_t weigh_u64(uint64_t w) { return w; }

// In-tile step of a two-level inverse CDF: wavefront 0 scans the n <= 128 integer weights w[i]
// of tile pk.i (ids 128 pk.i + i, held in LDS), two per lane, and returns to every thread the
// smallest id whose cumulative weight after pk.before exceeds pk.T (-1 if none: unreachable when
// the tile sums are those of the weights). `lds` must hold 8 uint64.
__device__ __forceinline__ int pick_in_tile(const uint64_t* w, int n, const Pick& pk,
                                            uint64_t* lds) {
  if (threadIdx.x < 64) {
    const int lane = lane_id();
    const uint64_t q0 = 2 * lane < n ? w[2 * lane] : 0;
    const uint64_t q1 = 2 * lane + 1 < n ? w[2 * lane + 1] : 0;
    const uint64_t in = wave_incl_scan_u64(q0 + q1);
    const bool h0 = pk.before + in - q1 > pk.T, h1 = pk.before + in > pk.T;
    const uint64_t hit = __ballot(h0 || h1);
    const int l = hit ? __ffsll(static_cast<unsigned long long>(hit)) - 1 : 0;
    const int pick0 = __shfl(static_cast<int>(h0), l);  // whole wavefront active
    if (lane == 0)
      lds[6] = hit ? static_cast<uint64_t>(static_cast<int64_t>(pk.i) * kTile + 2 * l +
                                           (pick0 ? 0 : 1))
                   : ~0ull;
  }
  __syncthreads();
  const uint64_t res = lds[6];
  __syncthreads();
  return res == ~0ull ? -1 : static_cast<int>(res);
}

// Two-level inverse CDF over per-tile integer sums by a whole 256-thread workgroup (every thread
// calls it): pick_block finds the tile holding the threshold, then wavefront 0 evaluates
// weight(v) for the tile's ids (v < V) into LDS and scans them.
template <class WeightFn>
__device__ int select_by_tiles_block(const uint64_t* tiles, int nT, int64_t V, uint32_t r,
                                     WeightFn weight, uint64_t* lds) {
  __shared__ uint64_t s_wt[kTile];
  const Pick pk = pick_block(nT, [&](int t) { return tiles[t]; }, weigh_u64, r, lds);
  if (pk.i < 0) return -1;
  const int64_t v0 = static_cast<int64_t>(pk.i) * kTile;
  const int n = static_cast<int>(V - v0 < kTile ? V - v0 : kTile);
  if (threadIdx.x < 64) {
    const int lane = lane_id();
    if (2 * lane < n) s_wt[2 * lane] = weight(v0 + 2 * lane);
    if (2 * lane + 1 < n) s_wt[2 * lane + 1] = weight(v0 + 2 * lane + 1);
  }
  __syncthreads();
  return pick_in_tile(s_wt, n, pk, lds);
}

}  // namespace dbl
