// Target-side sampling transform and early-determinism estimate.
//
// filter   one 1024-thread workgroup per row: the target's logits divided by the temperature,
//          restricted by top-k and then top-p, renormalised; -inf outside the kept set. Both cuts
//          are exact radix selections over order-preserving 32-bit keys of s = fl32(logit / T)
//          (four 8-bit digit passes with LDS histograms): by count for top-k (every value equal
//          to the k-th largest is kept), by the determinism contract's integer masses
//          floor(detexp32(fl32(s - max)) 2^40) for top-p, where tokens are taken by decreasing s
//          and, among equal s, increasing id, while the mass before them is below
//          ceil(p * total). Integer histograms make the kept set independent of summation order.
//          Temperature 0 keeps the lowest-index maximum only.
// early_determinism   per sampled block, (1/b) sum_j prod_{i<=j} p(x_i); the estimate is their
//          mean (appendix "Target-Block Early Determinism").
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "contract.hpp"
#include "kernels.hpp"
#include "wave.hpp"

namespace dbl {
namespace {

constexpr int kFT = 1024;  // threads per row
constexpr int kFW = kFT / 64;

__device__ __forceinline__ uint32_t order_key(float x) {
  const uint32_t u = __float_as_uint(x + 0.0f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Workgroup reductions over kFT threads (every thread calls them).
__device__ __forceinline__ uint64_t block_sum_u64(uint64_t v, uint64_t* red) {
  v = wave_sum_u64(v);
  if (lane_id() == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t s = 0;
#pragma unroll
  for (int w = 0; w < kFW; ++w) s += red[w];
  __syncthreads();
  return s;
}

__device__ __forceinline__ double block_sum_f64(double v, double* red) {
  v = wave_sum_f64(v);
  if (lane_id() == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int w = 0; w < kFW; ++w) s += red[w];
  __syncthreads();
  return s;
}

__device__ __forceinline__ uint64_t block_max_u64(uint64_t v, uint64_t* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t t = __shfl_xor(v, o);
    v = t > v ? t : v;
  }
  if (lane_id() == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t m = 0;
#pragma unroll
  for (int w = 0; w < kFW; ++w) m = red[w] > m ? red[w] : m;
  __syncthreads();
  return m;
}

// Picks, from a 256-bin histogram of the current digit (largest digit first), the digit whose
// bin holds the `need`-th unit counted from the top; returns it and what lies in larger digits.
__device__ __forceinline__ void pick_digit(const uint64_t* hist, uint64_t need, uint32_t* digit,
                                           uint64_t* above, uint32_t* sh_digit,
                                           uint64_t* sh_above) {
  if (threadIdx.x == 0) {
    uint64_t acc = 0;
    int d = 255;
    for (; d > 0; --d) {
      if (acc + hist[d] >= need) break;
      acc += hist[d];
    }
    *sh_digit = static_cast<uint32_t>(d);
    *sh_above = acc;
  }
  __syncthreads();
  *digit = *sh_digit;
  *above = *sh_above;
  __syncthreads();
}

__global__ __launch_bounds__(kFT) void filter_kernel(FilterArgs a) {
  __shared__ uint64_t hist[256];
  __shared__ uint64_t red[kFW];
  __shared__ double redd[kFW];
  __shared__ uint32_t sh_digit;
  __shared__ uint64_t sh_above;
  const int64_t n = blockIdx.x;
  const int64_t V = a.V;
  const float* in = a.logits + n * V;
  float* out = a.logp + n * V;
  const int tid = threadIdx.x;

  if (a.temperature == 0.0f) {  // lowest-index maximum
    uint64_t best = 0;
    for (int64_t v = tid; v < V; v += kFT) {
      const uint64_t k = (static_cast<uint64_t>(order_key(in[v])) << 32) |
                         (0xFFFFFFFFu - static_cast<uint32_t>(v));
      best = k > best ? k : best;
    }
    best = block_max_u64(best, red);
    const int64_t arg = 0xFFFFFFFFu - static_cast<uint32_t>(best);
    for (int64_t v = tid; v < V; v += kFT) out[v] = v == arg ? 0.0f : -INFINITY;
    return;
  }
  const float T = a.temperature;
  auto s_of = [&](int64_t v) { return __fdiv_rn(in[v], T); };

  // Row maximum (key of the largest s).
  uint64_t mk = 0;
  for (int64_t v = tid; v < V; v += kFT) {
    const uint64_t k = order_key(s_of(v));
    mk = k > mk ? k : mk;
  }
  const uint32_t max_key = static_cast<uint32_t>(block_max_u64(mk, red));
  const float m = __uint_as_float((max_key & 0x80000000u) ? (max_key & 0x7FFFFFFFu) : ~max_key);

  // Top-k: the k-th largest key, by count.
  uint32_t tk = 0;  // keep keys >= tk
  if (a.top_k > 0 && a.top_k < V) {
    uint32_t prefix = 0, pmask = 0;
    uint64_t need = static_cast<uint64_t>(a.top_k);
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = tid; i < 256; i += kFT) hist[i] = 0;
      __syncthreads();
      for (int64_t v = tid; v < V; v += kFT) {
        const uint32_t k = order_key(s_of(v));
        if ((k & pmask) == prefix) atomicAdd(reinterpret_cast<unsigned long long*>(&hist[(k >> shift) & 255]), 1ull);
      }
      __syncthreads();
      uint32_t d;
      uint64_t above;
      pick_digit(hist, need, &d, &above, &sh_digit, &sh_above);
      need -= above;
      prefix |= d << shift;
      pmask |= 255u << shift;
    }
    tk = prefix;
  }

  // Top-p: the crossing key by integer mass, then how many of the tokens at it are kept.
  uint32_t tp = 0;          // keep keys > tp, and the first n_tie tokens with key == tp
  uint64_t n_tie = ~0ull;
  if (a.top_p < 1.0f) {
    auto mass = [&](int64_t v, uint32_t k) -> uint64_t {
      return k >= tk ? quant40(detexp32(__fsub_rn(s_of(v), m))) : 0;
    };
    uint32_t prefix = 0, pmask = 0;
    uint64_t need = 0, tie_mass = 0;
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = tid; i < 256; i += kFT) hist[i] = 0;
      __syncthreads();
      for (int64_t v = tid; v < V; v += kFT) {
        const uint32_t k = order_key(s_of(v));
        if ((k & pmask) == prefix) {
          const uint64_t P = mass(v, k);
          if (P) atomicAdd(reinterpret_cast<unsigned long long*>(&hist[(k >> shift) & 255]),
                           static_cast<unsigned long long>(P));
        }
      }
      __syncthreads();
      if (shift == 24) {  // total mass of the kept set: T_p = ceil(p Z)
        uint64_t z = 0;
        for (int i = 0; i < 256; ++i) z += hist[i];
        need = static_cast<uint64_t>(ceil(__dmul_rn(static_cast<double>(a.top_p),
                                                    static_cast<double>(z))));
        if (need == 0) need = 1;
      }
      uint32_t d;
      uint64_t above;
      pick_digit(hist, need, &d, &above, &sh_digit, &sh_above);
      need -= above;
      if (shift == 0) tie_mass = hist[d];
      prefix |= d << shift;
      pmask |= 255u << shift;
    }
    tp = prefix;
    // Every token at key tp has the same mass; count how many of them there are.
    uint64_t cnt = 0;
    for (int64_t v = tid; v < V; v += kFT) cnt += order_key(s_of(v)) == tp ? 1 : 0;
    cnt = block_sum_u64(cnt, red);
    const uint64_t each = tie_mass / cnt;
    n_tie = (need + each - 1) / each;  // tokens at tp needed to reach T_p
    if (n_tie >= cnt) n_tie = ~0ull;
  }

  // Rank among the tokens at key tp (increasing id) when only some of them are kept: each
  // thread owns a contiguous run of ids.
  const int64_t per = (V + kFT - 1) / kFT;
  const int64_t r0 = min(V, tid * per), r1 = min(V, r0 + per);
  uint64_t tie_before = 0;
  if (n_tie != ~0ull) {
    uint64_t c = 0;
    for (int64_t v = r0; v < r1; ++v) c += order_key(s_of(v)) == tp ? 1 : 0;
    // exclusive scan of c over threads
    uint64_t incl = wave_incl_scan_u64(c);
    if (lane_id() == 63) red[tid >> 6] = incl;
    __syncthreads();
    uint64_t base = 0;
    for (int w = 0; w < (tid >> 6); ++w) base += red[w];
    __syncthreads();
    tie_before = base + incl - c;
  }
  auto kept = [&](int64_t v, uint32_t k, uint64_t rank) {
    if (k < tk) return false;
    if (a.top_p < 1.0f) {
      if (k < tp) return false;
      if (k == tp && n_tie != ~0ull && rank >= n_tie) return false;
    }
    return true;
  };

  // Normaliser over the kept set, then the output row: strided (coalesced) passes unless only
  // some of the tokens at the top-p cut are kept, which needs the id-ordered runs.
  auto pass = [&](auto fn) {
    if (n_tie == ~0ull) {
      for (int64_t v = tid; v < V; v += kFT) fn(v, 0ull);
    } else {
      uint64_t rank = tie_before;
      for (int64_t v = r0; v < r1; ++v) {
        fn(v, rank);
        if (order_key(s_of(v)) == tp) ++rank;
      }
    }
  };
  double se = 0.0;
  pass([&](int64_t v, uint64_t rank) {
    const float s = s_of(v);
    if (kept(v, order_key(s), rank)) se += exp(static_cast<double>(s) - static_cast<double>(m));
  });
  const double lse = log(block_sum_f64(se, redd));
  pass([&](int64_t v, uint64_t rank) {
    const float s = s_of(v);
    out[v] = kept(v, order_key(s), rank)
                 ? static_cast<float>(static_cast<double>(s) - static_cast<double>(m) - lse)
                 : -INFINITY;
  });
}

// Per sampled block: (1/b) sum_j prod_{i<=j} p(x_i); one thread per block.
__global__ __launch_bounds__(256) void determinism_terms_kernel(DeterminismArgs a) {
  const int64_t mblk = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (mblk >= a.M) return;
  double prod = 1.0, sum = 0.0;
  for (int64_t i = 0; i < a.b; ++i) {
    const int32_t x = a.x[mblk * a.b + i];
    const double lp = x >= 0 && x < a.V
                          ? static_cast<double>(a.logp[(mblk * a.b + i) * a.V + x])
                          : -INFINITY;
    prod *= exp(lp);
    sum += prod;
  }
  a.terms[mblk] = static_cast<float>(sum / static_cast<double>(a.b));
}

// Mean of the per-block terms in a fixed order (one workgroup).
__global__ __launch_bounds__(kFT) void determinism_mean_kernel(DeterminismArgs a) {
  __shared__ double redd[kFW];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < a.M; i += kFT) s += static_cast<double>(a.terms[i]);
  s = block_sum_f64(s, redd);
  if (threadIdx.x == 0) *a.mean = static_cast<float>(s / static_cast<double>(a.M));
}

}  // namespace

hipError_t launch_filter(const FilterArgs& a, hipStream_t stream) {
  if (a.N > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(filter_kernel, dim3(static_cast<unsigned>(a.N)), dim3(kFT), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_determinism(const DeterminismArgs& a, hipStream_t stream) {
  const int64_t blocks = (a.M + 255) / 256;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(determinism_terms_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !a.mean) return e;
  hipLaunchKernelGGL(determinism_mean_kernel, dim3(1), dim3(kFT), 0, stream, a);
  return hipGetLastError();
}

}  // namespace dbl
