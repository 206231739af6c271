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

// Calls fn(v, logit(v)) for every id of the row. When the row is 16-byte aligned and V is a
// multiple of 4 the loads are float4, issued kB at a time per thread so that one workgroup keeps
// enough bytes in flight to stream its row.
constexpr int kBatch = 8;

template <int kB = kBatch, class F>
__device__ __forceinline__ void row_scan_raw(const float* in, int64_t V, bool vec, F fn) {
  if (vec) {
    const float4* in4 = reinterpret_cast<const float4*>(in);
    const int64_t n4 = V >> 2;
    auto one = [&](int64_t j, const float4& x) {
      fn(4 * j, x.x);
      fn(4 * j + 1, x.y);
      fn(4 * j + 2, x.z);
      fn(4 * j + 3, x.w);
    };
    int64_t j = threadIdx.x;
    for (; j + (kB - 1) * kFT < n4; j += kB * kFT) {
      float4 x[kB];
#pragma unroll
      for (int u = 0; u < kB; ++u) x[u] = in4[j + u * kFT];
#pragma unroll
      for (int u = 0; u < kB; ++u) one(j + u * kFT, x[u]);
    }
    for (; j < n4; j += kFT) one(j, in4[j]);
  } else {
    for (int64_t v = threadIdx.x; v < V; v += kFT) fn(v, in[v]);
  }
}

// As row_scan_raw, with fn(v, s(v)), s(v) = fl32(logit(v) / T).
template <int kB = kBatch, class F>
__device__ __forceinline__ void row_scan(const float* in, int64_t V, float T, bool vec, F fn) {
  row_scan_raw<kB>(in, V, vec, [&](int64_t v, float x) { fn(v, __fdiv_rn(x, T)); });
}

__device__ __forceinline__ float key_value(uint32_t x) {
  return __uint_as_float((x & 0x80000000u) ? (x & 0x7FFFFFFFu) : ~x);
}

constexpr uint32_t kKeyNegInf = 0x007FFFFFu;  // order_key(-inf)
constexpr uint32_t kKeyPosInf = 0xFF800000u;  // order_key(+inf)

// Rounded division by T > 0 is monotone (non-decreasing) in the dividend, so the logits x with
// fl32(x / T) >= s form an upper set in key order. Returns its least key: a bisection over the
// keys of the non-NaN floats, every thread computing the same value.
__device__ __forceinline__ uint32_t least_logit_key(uint32_t s_key, float T) {
  auto ok = [&](uint32_t k) { return order_key(__fdiv_rn(key_value(k), T)) >= s_key; };
  if (ok(kKeyNegInf)) return kKeyNegInf;
  uint32_t lo = kKeyNegInf, hi = kKeyPosInf;  // ok(lo) false, ok(hi) true
  while (hi - lo > 1) {
    const uint32_t mid = lo + (hi - lo) / 2;
    if (ok(mid)) hi = mid; else lo = mid;
  }
  return hi;
}

// Sort key of a token: key(s) in the high word, ~id in the low word, so that a descending order
// visits tokens by decreasing s and, among equal s, increasing id.
__device__ __forceinline__ uint64_t visit_key(uint32_t key, int64_t v) {
  return (static_cast<uint64_t>(key) << 32) | (0xFFFFFFFFu - static_cast<uint32_t>(v));
}

// k-th largest of the 64 x 4 keys held by a wavefront (k <= 256): the largest t with at least k
// of them >= t, by bisection with ballots; no LDS, no barrier.
__device__ __forceinline__ uint32_t wave_kth_largest(uint32_t t0, uint32_t t1, uint32_t t2,
                                                     uint32_t t3, int k) {
  uint64_t lo = 0, hi = 0xFFFFFFFFu;  // count(>= lo) >= k always (every key is >= 0)
  while (lo < hi) {
    const uint64_t mid = lo + (hi - lo + 1) / 2;
    const uint32_t m32 = static_cast<uint32_t>(mid);
    const int c = __popcll(__ballot(t0 >= m32)) + __popcll(__ballot(t1 >= m32)) +
                  __popcll(__ballot(t2 >= m32)) + __popcll(__ballot(t3 >= m32));
    if (c >= k) lo = mid; else hi = mid - 1;
  }
  return static_cast<uint32_t>(lo);
}

// Fast path for top-k (0 < k <= kFastK < V): one streaming read and one streaming write of the
// row (fl32(x / T) is monotone in x, so selections on s are made on the logits' keys and only
// candidates are divided):
//   1. every thread writes -inf over its part of the output row and keeps the four largest logit
//      keys it sees;
//   2. a lower bound t of the row's k-th largest key: the largest over wavefronts of each
//      wavefront's k-th largest held key (k <= 256), else the k-th largest of all 4096 held keys
//      (workgroup bisection); each is the k-th largest of part of the row;
//   3. only threads holding a key >= x_low = least_logit_key(fl32(t / T)) can own a token with
//      s >= fl32(t / T) (their other logits are below their fourth largest); they re-read their
//      own ids and append every such token, with its s, to an LDS list;
//   4. the list is sorted in visiting order (s descending, id ascending); both cuts and the
//      normaliser follow from it, and the kept tokens' log-probabilities overwrite the -inf.
// Returns false (the caller then runs the radix path, which rewrites the whole row) if the list
// would overflow LDS.
constexpr int kFastK = 1024;
constexpr int kCandCap = 4096;

// Sorts a candidate list - visiting keys (key of s, ~id) of every token whose s is at least a
// lower bound of the row's k-th largest s - in visiting order (s descending, id ascending),
// applies both cuts and writes the kept tokens' log-probabilities; the rest of the output row
// already holds -inf. Needs n >= k and n <= kCandCap; all kFT threads call it.
// Sorts cand[0, n) (n <= kCandCap) in descending order: a bitonic network over the list padded
// with zeros to a power of two (every visiting key has a nonzero low word, ids being below
// 2^32 - 1). All kFT threads call it; it ends with a barrier.
__device__ void block_sort_desc(uint64_t* cand, int n) {
  const int tid = threadIdx.x;
  int np = 64;
  while (np < n) np <<= 1;
  for (int i = n + tid; i < np; i += kFT) cand[i] = 0;
  __syncthreads();
  for (int size = 2; size <= np; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < (np >> 1); i += kFT) {
        const int i0 = 2 * i - (i & (stride - 1));  // the pair (i0, i0 + stride)
        const int i1 = i0 + stride;
        const bool desc = (i0 & size) == 0;
        const uint64_t x = cand[i0], y = cand[i1];
        if ((x < y) == desc) {
          cand[i0] = y;
          cand[i1] = x;
        }
      }
      __syncthreads();
    }
  }
}

// Wavefront 0 alone, when the tokens tied with or above the k-th largest s number at most 64
// (the usual case for small k): those nk tokens are gathered one per lane, sorted in visiting
// order with a register bitonic network, and both cuts and the normaliser are wavefront
// reductions, with no workgroup barrier. tk is the k-th largest key of the list.
__device__ void finish_small(const FilterArgs& a, float* out, uint64_t* cand, int n,
                             uint32_t tk, int nk) {
  const int lane = lane_id();
  // compact the nk entries with key >= tk to the front of the list, in list order (an entry
  // moves only towards the front, past entries this wavefront has already read)
  int base = 0;
  for (int i0 = 0; i0 < n; i0 += 64) {
    const int i = i0 + lane;
    const uint64_t c = i < n ? cand[i] : 0;
    const bool in = i < n && static_cast<uint32_t>(c >> 32) >= tk;
    const uint64_t msk = __ballot(in);
    if (in) cand[base + __popcll(msk & ((1ull << lane) - 1))] = c;
    base += __popcll(msk);
    asm volatile("" ::: "memory");
  }
  uint64_t e = lane < nk ? cand[lane] : 0;
  // bitonic sort, descending, of one entry per lane (empty lanes hold 0)
#pragma unroll
  for (int size = 2; size <= 64; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      const uint64_t o = __shfl_xor(e, stride);
      const bool desc = (lane & size) == 0;
      const bool lower = (lane & stride) == 0;
      e = (lower == desc) ? (e > o ? e : o) : (e < o ? e : o);
    }
  }
  const float sv = key_value(static_cast<uint32_t>(e >> 32));
  const float m = __shfl(sv, 0);
  int nkeep = nk;
  if (a.top_p < 1.0f) {
    const uint64_t P = lane < nk ? quant_detexp32(__fsub_rn(sv, m)) : 0;
    const uint64_t incl = wave_incl_scan_u64(P);
    const uint64_t z = __shfl(incl, 63);
    uint64_t tp = static_cast<uint64_t>(ceil(__dmul_rn(static_cast<double>(a.top_p),
                                                       static_cast<double>(z))));
    if (tp == 0) tp = 1;
    nkeep = __popcll(__ballot(lane < nk && incl - P < tp));
  }
  const double x = lane < nkeep ? exp(static_cast<double>(sv) - static_cast<double>(m)) : 0.0;
  const double lse = log(wave_sum_f64(x));
  if (lane < nkeep) {
    const int64_t v = 0xFFFFFFFFu - static_cast<uint32_t>(e);
    out[v] = static_cast<float>(static_cast<double>(sv) - static_cast<double>(m) - lse);
  }
}

__device__ void finish_candidates(const FilterArgs& a, float* out, uint64_t* cand, int n,
                                  uint64_t* red, double* redd, int* sh_n) {
  const int tid = threadIdx.x;
  const int k = static_cast<int>(a.top_k);
  // Wavefront 0: the k-th largest key of the list (bisection with ballots over the list) and
  // how many entries are at or above it.
  if (tid < 64) {
    uint64_t lo = 0, hi = 0xFFFFFFFFu;
    int c = 0;
    if (n <= 8 * 64) {  // up to 8 keys per lane, in registers; counts by ballot
      uint32_t kk[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int i = tid + 64 * j;
        kk[j] = i < n ? static_cast<uint32_t>(cand[i] >> 32) : 0;
      }
      auto count = [&](uint32_t t) {
        int r = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) r += __popcll(__ballot(kk[j] >= t && tid + 64 * j < n));
        return r;
      };
      while (lo < hi) {
        const uint64_t mid = lo + (hi - lo + 1) / 2;
        if (count(static_cast<uint32_t>(mid)) >= k) lo = mid; else hi = mid - 1;
      }
      c = count(static_cast<uint32_t>(lo));
    } else {
      auto count = [&](uint64_t t) {
        int r = 0;
        for (int i = tid; i < n; i += 64) r += static_cast<uint32_t>(cand[i] >> 32) >= t ? 1 : 0;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) r += __shfl_xor(r, o);
        return r;
      };
      while (lo < hi) {
        const uint64_t mid = lo + (hi - lo + 1) / 2;
        if (count(mid) >= k) lo = mid; else hi = mid - 1;
      }
      c = count(lo);
    }
    if (tid == 0) {
      red[0] = lo;
      red[1] = static_cast<uint64_t>(c);
    }
  }
  __syncthreads();
  const uint32_t tk0 = static_cast<uint32_t>(red[0]);
  const int nk0 = static_cast<int>(red[1]);
  __syncthreads();
  if (nk0 <= 64) {
    if (tid < 64) finish_small(a, out, cand, n, tk0, nk0);
    return;
  }
  block_sort_desc(cand, n);
  auto key_at = [&](int i) { return static_cast<uint32_t>(cand[i] >> 32); };
  const float m = key_value(key_at(0));
  // top-k: the first k entries and every later one tied with the k-th (n >= k: the list holds
  // every token at or above the row's k-th largest key)
  const uint32_t tk = key_at(k - 1);
  int nk = k;
  while (nk < n && key_at(nk) >= tk) ++nk;
  int nkeep = nk;
  if (a.top_p < 1.0f) {
    // integer masses of the first nk entries, four per thread in list order; a token is kept
    // while the mass before it is below T_p = ceil(p Z)
    uint64_t P[4], loc = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = 4 * tid + j;
      P[j] = i < nk ? quant_detexp32(__fsub_rn(key_value(key_at(i)), m)) : 0;
      loc += P[j];
    }
    const uint64_t incl = wave_incl_scan_u64(loc);
    if (lane_id() == 63) red[tid >> 6] = incl;
    __syncthreads();
    uint64_t base = 0, z = 0;
#pragma unroll
    for (int w = 0; w < kFW; ++w) {
      const uint64_t r = red[w];
      base += w < (tid >> 6) ? r : 0;
      z += r;
    }
    __syncthreads();
    uint64_t tp = static_cast<uint64_t>(ceil(__dmul_rn(static_cast<double>(a.top_p),
                                                       static_cast<double>(z))));
    if (tp == 0) tp = 1;
    uint64_t before = base + incl - loc;
    uint64_t c = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (4 * tid + j < nk) {
        c += before < tp ? 1 : 0;
        before += P[j];
      }
    }
    nkeep = static_cast<int>(block_sum_u64(c, red));
  }
  double se = 0.0;
  for (int i = tid; i < nkeep; i += kFT)
    se += exp(static_cast<double>(key_value(key_at(i))) - static_cast<double>(m));
  const double lse = log(block_sum_f64(se, redd));
  // kept tokens (the first nkeep entries of the list)
  for (int i = tid; i < nkeep; i += kFT) {
    const uint64_t e = cand[i];
    const int64_t v = 0xFFFFFFFFu - static_cast<uint32_t>(e);
    out[v] = static_cast<float>(static_cast<double>(key_value(static_cast<uint32_t>(e >> 32))) -
                                static_cast<double>(m) - lse);
  }
}

__device__ bool filter_fast(const FilterArgs& a, const float* in, float* out, bool vec,
                            uint64_t* cand, int* resc, uint64_t* red, double* redd, int* sh_n,
                            int* sh_r) {
  const int tid = threadIdx.x;
  const int64_t V = a.V;
  const float T = a.temperature;
  const int k = static_cast<int>(a.top_k);
  // 1. -inf over the row; per-thread top-4 logit keys
  uint32_t t0 = 0, t1 = 0, t2 = 0, t3 = 0;
  auto insert = [&](float lv) {
    uint32_t x = order_key(lv);  // insertion into t0 >= t1 >= t2 >= t3, branch-free
    uint32_t y = max(t0, x);
    x = min(t0, x);
    t0 = y;
    y = max(t1, x);
    x = min(t1, x);
    t1 = y;
    y = max(t2, x);
    x = min(t2, x);
    t2 = y;
    t3 = max(t3, x);
  };
  if (vec) {
    const float4* in4 = reinterpret_cast<const float4*>(in);
    float4* out4 = reinterpret_cast<float4*>(out);
    const int64_t n4 = V >> 2;
    const float4 ninf = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
    int64_t j = tid;
    for (; j + (kBatch - 1) * kFT < n4; j += kBatch * kFT) {
      float4 x[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) x[u] = in4[j + u * kFT];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        out4[j + u * kFT] = ninf;
        insert(x[u].x);
        insert(x[u].y);
        insert(x[u].z);
        insert(x[u].w);
      }
    }
    for (; j < n4; j += kFT) {
      const float4 x = in4[j];
      out4[j] = ninf;
      insert(x.x);
      insert(x.y);
      insert(x.z);
      insert(x.w);
    }
  } else {
    for (int64_t v = tid; v < V; v += kFT) {
      insert(in[v]);
      out[v] = -INFINITY;
    }
  }
  // The kept tokens' values are stored later, possibly by other threads, over these -inf: wait
  // for this thread's stores before the barriers that follow.
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  // 2. lower bound of the row's k-th largest logit key
  uint32_t tlow;
  if (k <= 256) {
    tlow = static_cast<uint32_t>(block_max_u64(wave_kth_largest(t0, t1, t2, t3, k), red));
  } else {
    uint64_t lo = 0, hi = block_max_u64(t0, red);
    while (lo < hi) {
      const uint64_t mid = lo + (hi - lo + 1) / 2;
      const uint32_t m32 = static_cast<uint32_t>(mid);
      const uint32_t c = __popcll(__ballot(t0 >= m32)) + __popcll(__ballot(t1 >= m32)) +
                         __popcll(__ballot(t2 >= m32)) + __popcll(__ballot(t3 >= m32));
      if (lane_id() == 0) red[tid >> 6] = c;
      __syncthreads();
      uint64_t tot = 0;
#pragma unroll
      for (int w = 0; w < kFW; ++w) tot += red[w];
      __syncthreads();
      if (tot >= static_cast<uint64_t>(k)) lo = mid; else hi = mid - 1;
    }
    tlow = static_cast<uint32_t>(lo);
  }
  const uint32_t s_low = order_key(__fdiv_rn(key_value(tlow), T));
  const uint32_t x_low = least_logit_key(s_low, T);
  // 3. candidates from the threads that hold a key >= x_low: their ids are re-read by the whole
  //    workgroup (item w = (listed thread w / G, its w % G-th load), G loads per thread)
  if (tid == 0) {
    *sh_n = 0;
    *sh_r = 0;
  }
  __syncthreads();
  if (t0 >= x_low) resc[atomicAdd(sh_r, 1)] = tid;
  __syncthreads();
  const int nr = *sh_r;
  const int64_t units = vec ? (V >> 2) : V;              // float4 groups or single ids
  const int G = static_cast<int>((units + kFT - 1) / kFT);  // loads per thread, at most
  const int64_t items = static_cast<int64_t>(nr) * G;
  auto take = [&](int64_t v, float lv) {
    if (order_key(lv) >= x_low) {
      const int slot = atomicAdd(sh_n, 1);
      if (slot < kCandCap) cand[slot] = visit_key(order_key(__fdiv_rn(lv, T)), v);
    }
  };
  for (int64_t w0 = tid; w0 < items; w0 += kBatch * kFT) {
    int64_t jj[kBatch];
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int64_t w = w0 + static_cast<int64_t>(b) * kFT;
      const int64_t j = w < items ? resc[w / G] + (w % G) * static_cast<int64_t>(kFT) : units;
      jj[b] = j < units ? j : -1;
    }
    if (vec) {
      const float4* in4 = reinterpret_cast<const float4*>(in);
      float4 x[kBatch];
#pragma unroll
      for (int b = 0; b < kBatch; ++b) x[b] = jj[b] >= 0 ? in4[jj[b]] : make_float4(0, 0, 0, 0);
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        if (jj[b] < 0) continue;
        take(4 * jj[b], x[b].x);
        take(4 * jj[b] + 1, x[b].y);
        take(4 * jj[b] + 2, x[b].z);
        take(4 * jj[b] + 3, x[b].w);
      }
    } else {
      float x[kBatch];
#pragma unroll
      for (int b = 0; b < kBatch; ++b) x[b] = jj[b] >= 0 ? in[jj[b]] : 0.0f;
#pragma unroll
      for (int b = 0; b < kBatch; ++b)
        if (jj[b] >= 0) take(jj[b], x[b]);
    }
  }
  __syncthreads();
  const int n = *sh_n;
  __syncthreads();
  if (n > kCandCap) return false;
  finish_candidates(a, out, cand, n, red, redd, sh_n);
  return true;
}

// General path: exact radix selections over the keys of s (every k, and the nucleus alone),
// reading the row several times and writing all of it.
__device__ void filter_general(const FilterArgs& a, const float* in, float* out, bool vec,
                               uint64_t* hist, uint64_t* red, double* redd, uint32_t* sh_digit,
                               uint64_t* sh_above) {
  const int tid = threadIdx.x;
  const int64_t V = a.V;
  const float T = a.temperature;
  auto s_of = [&](int64_t v) { return __fdiv_rn(in[v], T); };
  // Row maximum (key of the largest s).
  uint32_t mk = 0;
  row_scan<4>(in, V, T, vec, [&](int64_t, float sv) {
    const uint32_t k = order_key(sv);
    mk = k > mk ? k : mk;
  });
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
      row_scan<4>(in, V, T, vec, [&](int64_t, float sv) {
        const uint32_t k = order_key(sv);
        if ((k & pmask) == prefix)
          atomicAdd(reinterpret_cast<unsigned long long*>(&hist[(k >> shift) & 255]), 1ull);
      });
      __syncthreads();
      uint32_t d;
      uint64_t above;
      pick_digit(hist, need, &d, &above, sh_digit, sh_above);
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
    auto mass = [&](float sv, uint32_t k) -> uint64_t {
      return k >= tk ? quant_detexp32(__fsub_rn(sv, m)) : 0;
    };
    uint32_t prefix = 0, pmask = 0;
    uint64_t need = 0, tie_mass = 0;
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = tid; i < 256; i += kFT) hist[i] = 0;
      __syncthreads();
      row_scan<4>(in, V, T, vec, [&](int64_t, float sv) {
        const uint32_t k = order_key(sv);
        if ((k & pmask) == prefix) {
          const uint64_t P = mass(sv, k);
          if (P) atomicAdd(reinterpret_cast<unsigned long long*>(&hist[(k >> shift) & 255]),
                           static_cast<unsigned long long>(P));
        }
      });
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
      pick_digit(hist, need, &d, &above, sh_digit, sh_above);
      need -= above;
      if (shift == 0) tie_mass = hist[d];
      prefix |= d << shift;
      pmask |= 255u << shift;
    }
    tp = prefix;
    // Every token at key tp has the same mass; count how many of them there are.
    uint64_t cnt = 0;
    row_scan<4>(in, V, T, vec, [&](int64_t, float sv) { cnt += order_key(sv) == tp ? 1 : 0; });
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
      row_scan<4>(in, V, T, vec, [&](int64_t v, float sv) { fn(v, sv, 0ull); });
    } else {
      uint64_t rank = tie_before;
      for (int64_t v = r0; v < r1; ++v) {
        const float sv = s_of(v);
        fn(v, sv, rank);
        if (order_key(sv) == tp) ++rank;
      }
    }
  };
  double se = 0.0;
  pass([&](int64_t v, float s, uint64_t rank) {
    if (kept(v, order_key(s), rank)) se += exp(static_cast<double>(s) - static_cast<double>(m));
  });
  const double lse = log(block_sum_f64(se, redd));
  pass([&](int64_t v, float s, uint64_t rank) {
    out[v] = kept(v, order_key(s), rank)
                 ? static_cast<float>(static_cast<double>(s) - static_cast<double>(m) - lse)
                 : -INFINITY;
  });
}

// Nucleus alone (top_k off, p < 1): with m the row maximum, every token's integer mass
// P(v) = floor(detexp32(fl32(s - m)) 2^40) goes to one of kNucBins bins by
// floor((m - s) kNucScale), which is non-increasing in s, so bins are ordered like s and tokens
// of one bin are contiguous in visiting order. The bin where the running mass reaches
// T_p = ceil(p Z) is the only one whose tokens need ordering: they are gathered and sorted, and
// the cut is found in it. Tokens with P = 0 follow all positive masses, whose total Z >= T_p, so
// they are never kept. The normaliser is the kept integer mass times 2^-40, within 2^-40 per
// token plus detexp32's rounding of the binary64 sum of exp(s - m). Four reads and one write of
// the row. Returns false (nothing written) if the cut's bin holds more than kCandCap tokens.
constexpr int kNucBins = 2048;
constexpr float kNucScale = kNucBins / 27.8f;  // P(v) = 0 below s - m = -40 ln 2 = -27.73
// Every token of a bin <= kNucSureBin has s - m > -27.16, so detexp32 > 1.5e-12 > 2^-40 and
// P(v) >= 1: when the cut's bin is one of them, the later passes need only the bins.
constexpr int kNucSureBin = 2000;

__device__ bool filter_nucleus(const FilterArgs& a, const float* in, float* out, bool vec,
                               uint64_t* bins, uint64_t* cand, uint64_t* red, int* sh_n) {
  const int tid = threadIdx.x;
  const int64_t V = a.V;
  const float T = a.temperature;
  // 1. maximum (division by T is monotone: the largest s is that of the largest logit)
  uint32_t mk = 0;
  row_scan_raw<4>(in, V, vec, [&](int64_t, float lv) {
    const uint32_t x = order_key(lv);
    mk = x > mk ? x : mk;
  });
  const float m = __fdiv_rn(key_value(static_cast<uint32_t>(block_max_u64(mk, red))), T);
  // s = fl32(x / T); x / 1 is x exactly, so T = 1 needs no division
  auto scan = [&](auto fn) {
    if (T == 1.0f)
      row_scan_raw<2>(in, V, vec, fn);
    else
      row_scan<2>(in, V, T, vec, fn);
  };
  auto mass_bin = [&](float sv, uint64_t* P) {
    const float d = __fsub_rn(sv, m);
    *P = quant_detexp32(d);
    return min(kNucBins - 1, static_cast<int>(__fmul_rn(-d, kNucScale)));
  };
  // 2. integer mass per bin
  for (int i = tid; i < kNucBins; i += kFT) bins[i] = 0;
  __syncthreads();
  scan([&](int64_t, float sv) {
    uint64_t P;
    const int b = mass_bin(sv, &P);
    if (P) atomicAdd(reinterpret_cast<unsigned long long*>(&bins[b]), static_cast<unsigned long long>(P));
  });
  __syncthreads();
  // the crossing bin: exclusive prefix of the bin masses (two bins per thread)
  const uint64_t b0 = bins[2 * tid], b1 = bins[2 * tid + 1];
  const uint64_t loc = b0 + b1;
  const uint64_t incl = wave_incl_scan_u64(loc);
  if (lane_id() == 63) red[tid >> 6] = incl;
  __syncthreads();
  uint64_t base = 0, z = 0;
#pragma unroll
  for (int w = 0; w < kFW; ++w) {
    const uint64_t r = red[w];
    base += w < (tid >> 6) ? r : 0;
    z += r;
  }
  __syncthreads();
  uint64_t tp = static_cast<uint64_t>(ceil(__dmul_rn(static_cast<double>(a.top_p),
                                                     static_cast<double>(z))));
  if (tp == 0) tp = 1;
  const uint64_t ex0 = base + incl - loc, ex1 = ex0 + b0;  // mass before bins 2 tid, 2 tid + 1
  if (ex0 < tp && tp <= ex1) {
    red[0] = 2 * tid;
    red[1] = ex0;
  } else if (ex1 < tp && tp <= ex1 + b1) {
    red[0] = 2 * tid + 1;
    red[1] = ex1;
  }
  if (tid == 0) *sh_n = 0;
  __syncthreads();
  const int bstar = static_cast<int>(red[0]);
  const uint64_t before = red[1];
  __syncthreads();
  auto bin_of = [&](float sv) {
    return min(kNucBins - 1, static_cast<int>(__fmul_rn(-__fsub_rn(sv, m), kNucScale)));
  };
  const bool sure = bstar <= kNucSureBin;
  // 3. the crossing bin's tokens, then their order
  if (sure) {
    scan([&](int64_t v, float sv) {
      if (bin_of(sv) == bstar) {
        const int slot = atomicAdd(sh_n, 1);
        if (slot < kCandCap) cand[slot] = visit_key(order_key(sv), v);
      }
    });
  } else {
    scan([&](int64_t v, float sv) {
      uint64_t P;
      if (mass_bin(sv, &P) == bstar && P) {
        const int slot = atomicAdd(sh_n, 1);
        if (slot < kCandCap) cand[slot] = visit_key(order_key(sv), v);
      }
    });
  }
  __syncthreads();
  const int n = *sh_n;
  __syncthreads();
  if (n > kCandCap) return false;
  block_sort_desc(cand, n);
  // kept prefix of the bin: four entries per thread in visiting order
  uint64_t P4[4], l4 = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = 4 * tid + j;
    P4[j] = i < n ? quant_detexp32(__fsub_rn(key_value(static_cast<uint32_t>(cand[i] >> 32)), m)) : 0;
    l4 += P4[j];
  }
  const uint64_t inc4 = wave_incl_scan_u64(l4);
  if (lane_id() == 63) red[tid >> 6] = inc4;
  __syncthreads();
  uint64_t base4 = 0;
#pragma unroll
  for (int w = 0; w < kFW; ++w) base4 += w < (tid >> 6) ? red[w] : 0;
  __syncthreads();
  uint64_t run = before + base4 + inc4 - l4;
  uint64_t cnt = 0, kept_mass = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (4 * tid + j < n && run < tp) {
      ++cnt;
      kept_mass += P4[j];
    }
    run += P4[j];
  }
  const uint64_t nkeep = block_sum_u64(cnt, red);
  const uint64_t kmass = before + block_sum_u64(kept_mass, red);
  const uint64_t cut = cand[nkeep - 1];
  const double lse = log(static_cast<double>(kmass)) - 40.0 * 0.6931471805599453;
  // 4. output row
  if (sure) {
    scan([&](int64_t v, float sv) {
      const int b = bin_of(sv);
      const bool kept = b < bstar || (b == bstar && visit_key(order_key(sv), v) >= cut);
      out[v] = kept ? static_cast<float>(static_cast<double>(sv) - static_cast<double>(m) - lse)
                    : -INFINITY;
    });
  } else {
    scan([&](int64_t v, float sv) {
      uint64_t P;
      const int b = mass_bin(sv, &P);
      const bool kept = P && (b < bstar || (b == bstar && visit_key(order_key(sv), v) >= cut));
      out[v] = kept ? static_cast<float>(static_cast<double>(sv) - static_cast<double>(m) - lse)
                    : -INFINITY;
    });
  }
  return true;
}

__global__ __launch_bounds__(kFT) void filter_kernel(FilterArgs a) {
  __shared__ uint64_t hist[256];
  __shared__ uint64_t cand[kCandCap];
  __shared__ int resc[kFT];
  __shared__ int sh_n, sh_r;
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
  const bool vec = (V & 3) == 0 && (reinterpret_cast<uintptr_t>(in) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(out) & 15) == 0;
  if (a.top_k > 0 && a.top_k <= kFastK && a.top_k < V &&
      filter_fast(a, in, out, vec, cand, resc, red, redd, &sh_n, &sh_r))
    return;

  filter_general(a, in, out, vec, hist, red, redd, &sh_digit, &sh_above);
}

// Rows with the nucleus alone (T > 0, top_k off, p < 1): the binned path, or the general one
// when the cut's bin is too crowded.
__global__ __launch_bounds__(kFT) void filter_nucleus_kernel(FilterArgs a) {
  __shared__ uint64_t hist[256];
  __shared__ uint64_t nbins[kNucBins];
  __shared__ uint64_t cand[kCandCap];
  __shared__ int sh_n;
  __shared__ uint64_t red[kFW];
  __shared__ double redd[kFW];
  __shared__ uint32_t sh_digit;
  __shared__ uint64_t sh_above;
  const int64_t n = blockIdx.x;
  const int64_t V = a.V;
  const float* in = a.logits + n * V;
  float* out = a.logp + n * V;
  const bool vec = (V & 3) == 0 && (reinterpret_cast<uintptr_t>(in) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(out) & 15) == 0;
  if (filter_nucleus(a, in, out, vec, nbins, cand, red, &sh_n)) return;
  filter_general(a, in, out, vec, hist, red, redd, &sh_digit, &sh_above);
}

// Rows split over kFilterSegs workgroups (0 < k <= 256, with a workspace). A segment
// workgroup streams its share of the row once (writing -inf, keeping each thread's four
// largest logit keys), bounds its share's k-th largest key from below (the largest over its
// wavefronts of each wavefront's k-th largest held key), and appends every token of its share
// at or above that bound (in s) to the row's candidate lists in the workspace: the row's top-k
// tokens of that share are among them, the share's k-th largest being at most the row's. A
// merge workgroup per row then sorts the lists and writes the kept tokens. A list that
// overflows sends the row to the general path.
constexpr int kSegThreads = 512;
constexpr int kSegWaves = kSegThreads / 64;

__global__ __launch_bounds__(kSegThreads) void filter_seg_kernel(FilterArgs a) {
  __shared__ int resc[kSegThreads];
  __shared__ int sh_n, sh_r;
  __shared__ uint32_t redk[kSegWaves];
  const int64_t row = blockIdx.x / kFilterSegs;
  const int seg = static_cast<int>(blockIdx.x % kFilterSegs);
  const int tid = threadIdx.x;
  const int64_t V = a.V;
  const float T = a.temperature;
  const int k = static_cast<int>(a.top_k);
  const float* in = a.logits + row * V;
  float* out = a.logp + row * V;
  const bool vec = (V & 3) == 0 && (reinterpret_cast<uintptr_t>(in) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(out) & 15) == 0;
  // This workgroup's units (float4 groups, or single ids): [u0, u1), thread t owns
  // u0 + t + i * kSegThreads.
  const int64_t units = vec ? (V >> 2) : V;
  const int64_t per = (units + kFilterSegs - 1) / kFilterSegs;
  const int64_t u0 = min(units, seg * per), u1 = min(units, u0 + per);
  uint32_t t0 = 0, t1 = 0, t2 = 0, t3 = 0;
  auto insert = [&](float lv) {
    uint32_t x = order_key(lv);
    uint32_t y = max(t0, x);
    x = min(t0, x);
    t0 = y;
    y = max(t1, x);
    x = min(t1, x);
    t1 = y;
    y = max(t2, x);
    x = min(t2, x);
    t2 = y;
    t3 = max(t3, x);
  };
  if (vec) {
    const float4* in4 = reinterpret_cast<const float4*>(in);
    float4* out4 = reinterpret_cast<float4*>(out);
    const float4 ninf = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
    int64_t j = u0 + tid;
    for (; j + (kBatch - 1) * kSegThreads < u1; j += kBatch * kSegThreads) {
      float4 x[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) x[u] = in4[j + u * kSegThreads];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        out4[j + u * kSegThreads] = ninf;
        insert(x[u].x);
        insert(x[u].y);
        insert(x[u].z);
        insert(x[u].w);
      }
    }
    for (; j < u1; j += kSegThreads) {
      const float4 x = in4[j];
      out4[j] = ninf;
      insert(x.x);
      insert(x.y);
      insert(x.z);
      insert(x.w);
    }
  } else {
    for (int64_t v = u0 + tid; v < u1; v += kSegThreads) {
      insert(in[v]);
      out[v] = -INFINITY;
    }
  }
  // Lower bound of this share's k-th largest logit key.
  const uint32_t kw = wave_kth_largest(t0, t1, t2, t3, k);
  if (lane_id() == 0) redk[tid >> 6] = kw;
  if (tid == 0) {
    sh_n = 0;
    sh_r = 0;
  }
  __syncthreads();
  uint32_t tlow = 0;
#pragma unroll
  for (int w = 0; w < kSegWaves; ++w) tlow = max(tlow, redk[w]);
  const uint32_t x_low = least_logit_key(order_key(__fdiv_rn(key_value(tlow), T)), T);
  if (t0 >= x_low) resc[atomicAdd(&sh_r, 1)] = tid;
  __syncthreads();
  // Re-read the listed threads' units, spread over the workgroup.
  const int nr = sh_r;
  const int G = static_cast<int>((u1 - u0 + kSegThreads - 1) / kSegThreads);
  const int64_t items = static_cast<int64_t>(nr) * G;
  uint64_t* list = a.seg_cand + blockIdx.x * static_cast<int64_t>(kFilterSegCap);
  auto take = [&](int64_t v, float lv) {
    if (order_key(lv) >= x_low) {
      const int slot = atomicAdd(&sh_n, 1);
      if (slot < kFilterSegCap) list[slot] = visit_key(order_key(__fdiv_rn(lv, T)), v);
    }
  };
  for (int64_t w = tid; w < items; w += kSegThreads) {
    const int64_t j = u0 + resc[w / G] + (w % G) * static_cast<int64_t>(kSegThreads);
    if (j >= u1) continue;
    if (vec) {
      const float4 x = reinterpret_cast<const float4*>(in)[j];
      take(4 * j, x.x);
      take(4 * j + 1, x.y);
      take(4 * j + 2, x.z);
      take(4 * j + 3, x.w);
    } else {
      take(j, in[j]);
    }
  }
  __syncthreads();
  if (tid == 0) a.seg_count[blockIdx.x] = sh_n;
}

// One workgroup per row: the row's segment lists, merged and finished; or the general path
// when a list overflowed.
__global__ __launch_bounds__(kFT) void filter_merge_kernel(FilterArgs a) {
  __shared__ uint64_t hist[256];
  __shared__ uint64_t cand[kCandCap];
  __shared__ int sh_n;
  __shared__ uint64_t red[kFW];
  __shared__ double redd[kFW];
  __shared__ uint32_t sh_digit;
  __shared__ uint64_t sh_above;
  const int64_t row = blockIdx.x;
  const int64_t V = a.V;
  const float* in = a.logits + row * V;
  float* out = a.logp + row * V;
  int cnt[kFilterSegs], n = 0;
  bool over = false;
#pragma unroll
  for (int sgi = 0; sgi < kFilterSegs; ++sgi) {
    cnt[sgi] = a.seg_count[row * kFilterSegs + sgi];
    over = over || cnt[sgi] > kFilterSegCap;
    n += cnt[sgi];
  }
  if (over) {
    const bool vec = (V & 3) == 0 && (reinterpret_cast<uintptr_t>(in) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(out) & 15) == 0;
    filter_general(a, in, out, vec, hist, red, redd, &sh_digit, &sh_above);
    return;
  }
  int base = 0;
#pragma unroll
  for (int sgi = 0; sgi < kFilterSegs; ++sgi) {
    const uint64_t* list = a.seg_cand + (row * kFilterSegs + sgi) * static_cast<int64_t>(kFilterSegCap);
    for (int i = threadIdx.x; i < cnt[sgi]; i += kFT) cand[base + i] = list[i];
    base += cnt[sgi];
  }
  __syncthreads();
  finish_candidates(a, out, cand, n, red, redd, &sh_n);
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
  if (a.N > 0x7fffffff / kFilterSegs) return hipErrorInvalidConfiguration;
  const bool split = a.seg_cand && a.seg_count && a.temperature > 0.0f && a.top_k > 0 &&
                     a.top_k <= 256 && a.top_k < a.V && a.V >= kFilterSegs * 4096;
  const bool nucleus = a.temperature > 0.0f && (a.top_k == 0 || a.top_k >= a.V) &&
                       a.top_p < 1.0f;
  if (nucleus) {
    hipLaunchKernelGGL(filter_nucleus_kernel, dim3(static_cast<unsigned>(a.N)), dim3(kFT), 0,
                       stream, a);
    return hipGetLastError();
  }
  if (!split) {
    hipLaunchKernelGGL(filter_kernel, dim3(static_cast<unsigned>(a.N)), dim3(kFT), 0, stream, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(filter_seg_kernel, dim3(static_cast<unsigned>(a.N * kFilterSegs)),
                     dim3(kSegThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(filter_merge_kernel, dim3(static_cast<unsigned>(a.N)), dim3(kFT), 0, stream,
                     a);
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
