// Stochastic verification of DBLast blocks and the expected-accepted-length reduction.
//
//   chain     one wavefront per block, lane z = category. Walks the K positions in order:
//             category posterior w_{k,z} (Eq. category-posterior, in the log domain), the
//             prefix-marginalised proposal at the drafted token
//             q_k(x_k | x_<k) = sum_z w_{k,z} q_k(x_k | z) (Eq. dep-next-token-distribution),
//             the accept test u < p/q while all earlier positions were accepted
//             (Eq. accept-prob), and A_k = min(1, p/q) for AL_b (Eq. acceptance-length).
//             The posterior is kept for every position (workspace) because the acceptance mass
//             is needed along the whole draft.
//   beta      grid (position, vocabulary chunk), the HBM stream: reads the R branch rows and
//             the target row of every position once and sums min(p(v), sum_z w_z q_z(v)).
//   residual  grid (block, vocabulary chunk): integer tile sums of the residual
//             max(P - Q, 0) at the first rejected position (and of P for the fallback), or of
//             the bonus row when every position was accepted.
//   finalize  one 256-thread workgroup per block: acceptance masses,
//             E = sum_i prod_{j<=i} beta_j, and the residual/bonus inverse-CDF draw (the tile
//             from the tile sums, then the tile's weights staged in LDS in one round of loads).
//   stream    (verification with V % 4 == 0 and masses requested: the usual case) beta and
//             residual in one launch between the chain and finalize: the residual's tile sums
//             come from the stream's own loads at the first rejected position.
// The expected-length reduction along a given trajectory runs chain, beta and finalize (no
// accept test, no residual). Built with floating-point contraction off (determinism contract).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "contract.hpp"
#include "kernels.hpp"
#include "wave.hpp"

namespace dbl {
namespace {

__device__ __forceinline__ bool in_vocab(int32_t x, int64_t V) { return x >= 0 && x < V; }

__global__ __launch_bounds__(64) void chain_kernel(VerifyArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t b = blockIdx.x;
  const int lane = lane_id();
  const int R = static_cast<int>(k_.R);
  const uint64_t seq = static_cast<uint64_t>(k_.seq_offset + b);
  double L = prior_log_weight(k_.prior + b * k_.R, R, k_.z_temp);
  bool alive = true;
  int n_acc = 0;
  double prodA = 1.0, al = 0.0;
  for (int64_t k = 0; k < k_.K; ++k) {
    const double w = normalize_weight(L, R);
    const int64_t row = (b * k_.K + k) * k_.R + lane;
    if (lane < R) a.wpost[row] = w;
    const int32_t xk = a.x[b * k_.K + k];
    const bool ok = in_vocab(xk, k_.V);
    float lq = -INFINITY;
    if (ok && lane < R)
      lq = flat_lq(k_.tls[row * k_.V + xk], k_.lmass[row * k_.nT + xk / kTile], k_.lse[row]);
    L = __dadd_rn(L, static_cast<double>(lq));
    if (a.trajectory) continue;
    const double y = static_cast<double>(detexp32(lq));
    double Q = 0.0;
    for (int z = 0; z < R; ++z) Q = __dadd_rn(Q, __dmul_rn(lane_f64(w, z), lane_f64(y, z)));
    const double P = ok ? static_cast<double>(detexp32(a.logp[(b * a.Kp + k) * k_.V + xk])) : 0.0;
    const double A = Q > 0.0 ? fmin(1.0, P / Q) : (P > 0.0 ? 1.0 : 0.0);
    prodA = __dmul_rn(prodA, A);
    al = __dadd_rn(al, prodA);
    if (alive) {
      const uint32_t r = draw(k_.seed, kAccept, static_cast<uint32_t>(k), seq, k_.step);
      if (accept_int(r, quant40d(Q), quant40d(P)))
        ++n_acc;
      else
        alive = false;
    }
  }
  if (!a.trajectory && lane == 0) {
    a.n_accept[b] = n_acc;
    if (a.al) a.al[b] = static_cast<float>(al);
  }
}

// Parallel form of chain_kernel for K * R <= kChainMaxKR and K <= kChainMaxK (one workgroup
// per block). The posterior at position k depends only on the drafted prefix, not on the
// accept decisions, so every position is handled at once: thread (k, z) folds its own prefix
// L_{k,z} = (((L_{0,z} + lq_{0,z}) + lq_{1,z}) + ...) + lq_{k-1,z} in the same order as the
// sequential walk, a segment of lanes per position normalises it and forms q_k(x_k | x_<k)
// (eight positions per wavefront at R <= 8: the normalisation's serial steps were 56% of the
// kernel with one position per wavefront), and one wavefront then runs the integer accept chain
// over k. Bit-identical to chain_kernel.
constexpr int kChainMaxKR = 2048;
constexpr int kChainMaxK = 256;

__global__ __launch_bounds__(256) void chain_parallel_kernel(VerifyArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  const int R = static_cast<int>(k_.R);
  const int K = static_cast<int>(k_.K);
  const int KR = K * R;
  const uint64_t seq = static_cast<uint64_t>(k_.seq_offset + b);
  __shared__ float s_lq[kChainMaxKR];
  __shared__ double s_L[kChainMaxKR];
  __shared__ double s_L0[kMaxR];
  __shared__ double s_Q[kChainMaxK];
  __shared__ double s_P[kChainMaxK];
  uint32_t r_first = 0;  // wavefront 0: the accept draw of position lane (K R <= 256)
  bool have_r = false;
  if (KR <= static_cast<int>(blockDim.x)) {
    have_r = true;
    // At most one (k, z) per thread (every workload shape of the paper): the drafted tokens and
    // the prior, then the branch and target values at the tokens, each round of loads issued
    // together with clamped (in-bounds) indices before any value is used.
    const int i = min(tid, KR - 1), k = i / R, z = i % R, kp = min(tid, K - 1);
    const int32_t xk = a.x[b * k_.K + k], xp = a.x[b * k_.K + kp];
    const float pl = k_.prior[b * k_.R + min(lane, R - 1)];
    const bool okq = in_vocab(xk, k_.V), okp = in_vocab(xp, k_.V);
    const int64_t row = (b * k_.K + k) * k_.R + z, vq = okq ? xk : 0, vp = okp ? xp : 0;
    const float t = k_.tls[row * k_.V + vq], lm = k_.lmass[row * k_.nT + vq / kTile];
    const float ls = k_.lse[row], lp = a.logp[(b * a.Kp + kp) * k_.V + vp];
    // Wavefront 0's accept draws for positions 0..63, computed while the loads are in flight.
    if (wave == 0 && !a.trajectory)
      r_first = draw(k_.seed, kAccept, static_cast<uint32_t>(lane), seq, k_.step);
    if (wave == 0) {
      const double l0 = prior_log_weight_of(pl, R, k_.z_temp);
      if (lane < R) s_L0[lane] = l0;
    }
    if (tid < KR) s_lq[tid] = okq ? flat_lq(t, lm, ls) : -INFINITY;
    if (!a.trajectory && tid < K) s_P[tid] = okp ? static_cast<double>(detexp32(lp)) : 0.0;
  } else {
    if (wave == 0) {
      const double l0 = prior_log_weight(k_.prior + b * k_.R, R, k_.z_temp);
      if (lane < R) s_L0[lane] = l0;
    }
    for (int i = tid; i < KR; i += blockDim.x) {
      const int k = i / R, z = i % R;
      const int64_t row = (b * k_.K + k) * k_.R + z;
      const int32_t xk = a.x[b * k_.K + k];
      s_lq[i] = in_vocab(xk, k_.V) ? flat_lq(k_.tls[row * k_.V + xk],
                                             k_.lmass[row * k_.nT + xk / kTile], k_.lse[row])
                                   : -INFINITY;
    }
    if (!a.trajectory) {
      for (int k = tid; k < K; k += blockDim.x) {
        const int32_t xk = a.x[b * k_.K + k];
        s_P[k] = in_vocab(xk, k_.V)
                     ? static_cast<double>(detexp32(a.logp[(b * a.Kp + k) * k_.V + xk]))
                     : 0.0;
      }
    }
  }
  __syncthreads();
  for (int i = tid; i < KR; i += blockDim.x) {
    const int k = i / R, z = i % R;
    double L = s_L0[z];
    int j = 0;
    for (; j + 4 <= k; j += 4) {  // four LDS reads in flight; the additions stay in order
      const float q0 = s_lq[j * R + z], q1 = s_lq[(j + 1) * R + z];
      const float q2 = s_lq[(j + 2) * R + z], q3 = s_lq[(j + 3) * R + z];
      L = __dadd_rn(L, static_cast<double>(q0));
      L = __dadd_rn(L, static_cast<double>(q1));
      L = __dadd_rn(L, static_cast<double>(q2));
      L = __dadd_rn(L, static_cast<double>(q3));
    }
    for (; j < k; ++j) L = __dadd_rn(L, static_cast<double>(s_lq[j * R + z]));
    s_L[i] = L;
  }
  __syncthreads();
  // 64 / G positions per wavefront at a time, one segment of G lanes each (lane z = category).
  const int nwaves = blockDim.x >> 6;
  auto weights = [&](auto g_c) {
    constexpr int G = decltype(g_c)::value, P = 64 / G;
    const int seg = lane / G, z = lane % G;
    for (int k0 = wave * P; k0 < K; k0 += nwaves * P) {
      const int k = k0 + seg;
      const bool own = k < K && z < R;
      const double L = own ? s_L[k * R + z] : -INFINITY;
      const double w = normalize_weight_seg<G>(L, R);
      if (own) a.wpost[(b * k_.K + k) * k_.R + z] = w;
      if (!a.trajectory) {
        const double y = own ? static_cast<double>(detexp32(s_lq[k * R + z])) : 0.0;
        double Q = 0.0;
        if constexpr (G <= 16) {  // all shuffles in flight, then the ordered sum
          double wv[G], yv[G];
#pragma unroll
          for (int zz = 0; zz < G; ++zz) {
            wv[zz] = __shfl(w, seg * G + zz);
            yv[zz] = __shfl(y, seg * G + zz);
          }
#pragma unroll
          for (int zz = 0; zz < G; ++zz)
            if (zz < R) Q = __dadd_rn(Q, __dmul_rn(wv[zz], yv[zz]));
        } else {
          for (int zz = 0; zz < R; ++zz)
            Q = __dadd_rn(Q, __dmul_rn(__shfl(w, seg * G + zz), __shfl(y, seg * G + zz)));
        }
        if (k < K && z == 0) s_Q[k] = Q;
      }
    }
  };
  if (R <= 8)
    weights(std::integral_constant<int, 8>{});
  else if (R <= 16)
    weights(std::integral_constant<int, 16>{});
  else if (R <= 32)
    weights(std::integral_constant<int, 32>{});
  else
    weights(std::integral_constant<int, 64>{});
  if (a.trajectory) return;
  __syncthreads();
  // Wavefront 0: 64 positions' accept tests at a time (the draws do not depend on earlier
  // outcomes); n_accept is the index of the first rejection. The running product of the A_k is
  // taken in position order by every lane alike.
  if (wave == 0) {
    int n_acc = K;
    double prodA = 1.0, al = 0.0;
    for (int k0 = 0; k0 < K; k0 += 64) {
      const int k = k0 + lane;
      bool rej = false;
      double A = 0.0;
      if (k < K) {
        const double Q = s_Q[k], P = s_P[k];
        A = Q > 0.0 ? fmin(1.0, P / Q) : (P > 0.0 ? 1.0 : 0.0);
        const uint32_t r = k0 == 0 && have_r
                               ? r_first
                               : draw(k_.seed, kAccept, static_cast<uint32_t>(k), seq, k_.step);
        rej = !accept_int(r, quant40d(Q), quant40d(P));
      }
      const uint64_t rejm = __ballot(rej);
      if (rejm && n_acc == K) n_acc = k0 + __ffsll(static_cast<unsigned long long>(rejm)) - 1;
      const int kn = min(64, K - k0);
      for (int j = 0; j < kn; ++j) {
        prodA = __dmul_rn(prodA, lane_f64(A, j));
        al = __dadd_rn(al, prodA);
      }
    }
    if (lane == 0) {
      a.n_accept[b] = n_acc;
      if (a.al) a.al[b] = static_cast<float>(al);
    }
  }
}

// Acceptance-mass stream: workgroup (position, chunk of kTilesPerChunk vocabulary tiles).
// beta partial = sum_v min(p(v), sum_z w_z q_z(v)) over the chunk, with p = exp(logp) and
// q_z = exp(tls + lmass - lse) evaluated as exp2(tls * log2 e + o_z,t), the per-tile offsets
// o_z,t prepared once in LDS. Every row is streamed once with 16-byte loads; RT > 0 fixes the
// number of categories at compile time so all R + 1 loads of a step are in flight together.
constexpr float kLog2eF = 1.4426950408889634f;

template <int RT>
__device__ __forceinline__ void beta_body(const VerifyArgs& a, int64_t pos, int chunk,
                                          int nchunk) {
  const BlockArgs& k_ = a.blk;
  const int64_t b = pos / k_.K;
  const int64_t k = pos % k_.K;
  const int R = RT > 0 ? RT : static_cast<int>(k_.R);
  const int64_t V = k_.V;
  __shared__ float s_w[kMaxR];
  __shared__ float s_off[kMaxR][kTilesPerChunk];
  __shared__ float red[4];
  const int t0 = chunk * kTilesPerChunk;
  const int nt = min(kTilesPerChunk, k_.nT - t0);
  const int64_t m0 = pos * k_.R;
  for (int i = threadIdx.x; i < R * kTilesPerChunk; i += blockDim.x) {
    const int z = i / kTilesPerChunk, tt = i % kTilesPerChunk;
    if (tt < nt)
      s_off[z][tt] = (k_.lmass[(m0 + z) * k_.nT + t0 + tt] - k_.lse[m0 + z]) * kLog2eF;
  }
  if (threadIdx.x < R) s_w[threadIdx.x] = static_cast<float>(a.wpost[m0 + threadIdx.x]);
  __syncthreads();
  const int64_t vb = static_cast<int64_t>(t0) * kTile;
  const int64_t ve = min(V, vb + static_cast<int64_t>(nt) * kTile);
  const float* prow = a.logp + (b * a.Kp + k) * V;
  const float* trow = k_.tls + m0 * V;
  float acc = 0.0f;
  if ((V & 3) == 0) {
    for (int64_t v = vb + 4 * threadIdx.x; v < ve; v += 4 * blockDim.x) {
      const int tt = static_cast<int>((v - vb) >> 7);
      const float4 p = load_stream4(prow + v);
      float4 x[RT > 0 ? RT : 1];
      float q0 = 0.0f, q1 = 0.0f, q2 = 0.0f, q3 = 0.0f;
      if constexpr (RT > 0) {
#pragma unroll
        for (int z = 0; z < RT; ++z) x[z] = load_stream4(trow + z * V + v);
#pragma unroll
        for (int z = 0; z < RT; ++z) {
          const float o = s_off[z][tt], w = s_w[z];
          q0 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(x[z].x, kLog2eF, o)), q0);
          q1 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(x[z].y, kLog2eF, o)), q1);
          q2 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(x[z].z, kLog2eF, o)), q2);
          q3 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(x[z].w, kLog2eF, o)), q3);
        }
      } else {
        for (int z = 0; z < R; ++z) {
          const float4 xz = load_stream4(trow + z * V + v);
          const float o = s_off[z][tt], w = s_w[z];
          q0 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(xz.x, kLog2eF, o)), q0);
          q1 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(xz.y, kLog2eF, o)), q1);
          q2 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(xz.z, kLog2eF, o)), q2);
          q3 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(xz.w, kLog2eF, o)), q3);
        }
      }
      acc += fminf(__builtin_amdgcn_exp2f(p.x * kLog2eF), q0) +
             fminf(__builtin_amdgcn_exp2f(p.y * kLog2eF), q1) +
             fminf(__builtin_amdgcn_exp2f(p.z * kLog2eF), q2) +
             fminf(__builtin_amdgcn_exp2f(p.w * kLog2eF), q3);
    }
  } else {
    for (int64_t v = vb + threadIdx.x; v < ve; v += blockDim.x) {
      const int tt = static_cast<int>((v - vb) >> 7);
      float q = 0.0f;
      for (int z = 0; z < R; ++z)
        q = fmaf(s_w[z], __builtin_amdgcn_exp2f(fmaf(trow[z * V + v], kLog2eF, s_off[z][tt])), q);
      acc += fminf(__builtin_amdgcn_exp2f(prow[v] * kLog2eF), q);
    }
  }
  acc = wave_sum_f32(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0)
    a.beta_part[pos * nchunk + chunk] = (red[0] + red[1]) + (red[2] + red[3]);
}

template <int RT>
__global__ __launch_bounds__(256) void beta_kernel(VerifyArgs a) {
  beta_body<RT>(a, blockIdx.x, blockIdx.y, gridDim.y);
}

// Residual / bonus tile sums: workgroup (block, chunk of 32 vocabulary tiles), 8 lanes per
// tile, each lane 16 ids read with 16-byte loads. At the first rejected position ks the integer
// weights are P(v) = floor(detexp32(logp) 2^40) and R(v) = max(P(v) - Q(v), 0) with
// Q(v) = floor((sum over ascending z of w_z detexp32(lq_z(v))) 2^40); after full acceptance
// only P of the bonus row. RT > 0 fixes the number of categories at compile time.
template <int RT>
__device__ __forceinline__ void residual_body(const VerifyArgs& a, int64_t b, int chunk) {
  const BlockArgs& k_ = a.blk;
  const int ks = a.n_accept[b];
  const bool residual = ks < k_.K;
  if (!residual && a.Kp != k_.K + 1) return;
  const int R = RT > 0 ? RT : static_cast<int>(k_.R);
  __shared__ double wz[kMaxR];
  if (residual && threadIdx.x < R) wz[threadIdx.x] = a.wpost[(b * k_.K + ks) * k_.R + threadIdx.x];
  __syncthreads();
  const int sub = threadIdx.x & 7;
  const int t = chunk * kTilesPerChunk + (threadIdx.x >> 3);
  const int64_t V = k_.V;
  uint64_t sp = 0, sr = 0;
  if (t < k_.nT) {
    const int64_t v0 = static_cast<int64_t>(t) * kTile;
    const float* prow = a.logp + (b * a.Kp + ks) * V + v0;
    const int64_t m0 = (b * k_.K + (residual ? ks : 0)) * k_.R;
    float off[RT > 0 ? RT : 1];
    if constexpr (RT > 0) {
      if (residual) {
#pragma unroll
        for (int z = 0; z < RT; ++z)
          off[z] = __fsub_rn(k_.lmass[(m0 + z) * k_.nT + t], k_.lse[m0 + z]);
      }
    }
    auto weights = [&](int v, float pv, const float* tv, int tstride, uint64_t& P, uint64_t& Rw) {
      P = quant_detexp32(pv);
      Rw = 0;
      if (!residual) return;
      double Q = 0.0;
      if constexpr (RT > 0) {
#pragma unroll
        for (int z = 0; z < RT; ++z)
          Q = __dadd_rn(Q, __dmul_rn(wz[z], static_cast<double>(
                                                detexp32(__fadd_rn(tv[z * tstride], off[z])))));
      } else {
        for (int z = 0; z < R; ++z) {
          const float o = __fsub_rn(k_.lmass[(m0 + z) * k_.nT + t], k_.lse[m0 + z]);
          Q = __dadd_rn(Q, __dmul_rn(wz[z], static_cast<double>(
                                                detexp32(__fadd_rn(tv[z * tstride], o)))));
        }
      }
      const uint64_t Qi = quant40d(Q);
      Rw = P > Qi ? P - Qi : 0;
      (void)v;
    };
    const float* trow = k_.tls + m0 * V + v0;
    if ((V & 3) == 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int v = 4 * sub + 32 * i;
        if (v0 + v < V) {
          const float4 p4 = load_stream4(prow + v);
          const float pe[4] = {p4.x, p4.y, p4.z, p4.w};
          float4 x4[RT > 0 ? RT : 1];
          if constexpr (RT > 0) {
            if (residual) {
#pragma unroll
              for (int z = 0; z < RT; ++z)
                x4[z] = load_stream4(trow + z * V + v);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              uint64_t P, Rw;
              float tv[RT];
              if (residual) {
#pragma unroll
                for (int z = 0; z < RT; ++z)
                  tv[z] = e == 0 ? x4[z].x : e == 1 ? x4[z].y : e == 2 ? x4[z].z : x4[z].w;
              }
              weights(v + e, pe[e], tv, 1, P, Rw);
              sp += P;
              sr += Rw;
            }
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              uint64_t P, Rw;
              weights(v + e, pe[e], trow + v + e, static_cast<int>(V), P, Rw);
              sp += P;
              sr += Rw;
            }
          }
        }
      }
    } else {
      for (int i = 0; i < 16; ++i) {
        const int v = sub + 8 * i;
        if (v0 + v < V) {
          uint64_t P, Rw;
          if constexpr (RT > 0) {
            float tv[RT];
            if (residual) {
#pragma unroll
              for (int z = 0; z < RT; ++z) tv[z] = trow[z * V + v];
            }
            weights(v, prow[v], tv, 1, P, Rw);
          } else {
            weights(v, prow[v], trow + v, static_cast<int>(V), P, Rw);
          }
          sp += P;
          sr += Rw;
        }
      }
    }
  }
  sp += __shfl_xor(sp, 1);
  sp += __shfl_xor(sp, 2);
  sp += __shfl_xor(sp, 4);
  sr += __shfl_xor(sr, 1);
  sr += __shfl_xor(sr, 2);
  sr += __shfl_xor(sr, 4);
  if (sub == 0 && t < k_.nT) {
    a.p_tiles[b * k_.nT + t] = sp;
    a.res_tiles[b * k_.nT + t] = sr;
  }
}

template <int RT>
__global__ __launch_bounds__(256) void residual_kernel(VerifyArgs a) {
  residual_body<RT>(a, blockIdx.x, blockIdx.y);
}

// Residual / bonus tile sums and the acceptance-mass stream in one launch: workgroups
// x < B are the residual's (issued first, so its ALU-heavy blocks overlap the stream), the rest
// the acceptance-mass stream's. The two write disjoint outputs.
template <int RT>
__global__ __launch_bounds__(256) void beta_residual_kernel(VerifyArgs a) {
  const int64_t B = a.blk.B;
  if (blockIdx.x < B)
    residual_body<RT>(a, blockIdx.x, blockIdx.y);
  else
    beta_body<RT>(a, blockIdx.x - B, blockIdx.y, gridDim.y);
}

// Block b: acceptance masses and E (binary64 sums of the chunk partials), then the residual or
// bonus draw by inverse CDF over the tile sums. Run by a whole 256-thread workgroup.
constexpr int kStageBatch = 8;  // loads in flight per thread when staging a tile's branch values

__device__ void finalize_block(const VerifyArgs& a, int64_t b, int nchunk) {
  __shared__ double s_beta[kChainMaxK];
  __shared__ uint64_t lds[8];
  __shared__ double wz[kMaxR];
  __shared__ uint64_t s_wt[kTile];         // integer weights of the selected tile
  __shared__ float s_y[kMaxR * kTile];     // detexp32 of the tile's branch log-probabilities
  const BlockArgs& k_ = a.blk;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  const int K = static_cast<int>(k_.K);
  __shared__ int s_ks;
  // The first rejected position, loaded together with the partials below (an LDS copy keeps the
  // load ahead of the reduction's barriers).
  if (!a.trajectory && tid == 0) s_ks = a.n_accept[b];
  if (a.beta || a.exp_len) {
    for (int k0 = 0; k0 < K; k0 += kChainMaxK) {
      const int kn = min(kChainMaxK, K - k0);
      // Four positions per wavefront at a time, their loads issued together with clamped
      // (in-bounds) indices before any is summed; each position's sum is taken in the same order
      // as one at a time: lane l adds chunks l, l + 64, ..., then a wavefront sum.
      for (int kk0 = 4 * wave; kk0 < kn; kk0 += 16) {
        double sum[4] = {0.0, 0.0, 0.0, 0.0};
        for (int c0 = 0; c0 < nchunk; c0 += 64) {  // one pass up to 64 chunks
          const int c = min(c0 + lane, nchunk - 1);
          float v[4];
#pragma unroll
          for (int u = 0; u < 4; ++u)
            v[u] = a.beta_part[(b * k_.K + k0 + min(kk0 + u, kn - 1)) * nchunk + c];
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (c0 + lane < nchunk) sum[u] += static_cast<double>(v[u]);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) sum[u] = wave_sum_f64(sum[u]);
        if (lane == 0) {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (kk0 + u < kn) s_beta[kk0 + u] = sum[u];
        }
      }
      __syncthreads();
      for (int kk = tid; kk < kn; kk += blockDim.x)
        if (a.beta) a.beta[b * k_.K + k0 + kk] = static_cast<float>(s_beta[kk]);
      if (a.exp_len && wave == 0) {
        // Running product and sum over all positions in order, kept in lds[7] / lds[6] across
        // chunks; every lane of wavefront 0 takes the same steps on values held in its lanes.
        double prod = k0 == 0 ? 1.0 : __longlong_as_double(static_cast<long long>(lds[7]));
        double E = k0 == 0 ? 0.0 : __longlong_as_double(static_cast<long long>(lds[6]));
        for (int c0 = 0; c0 < kn; c0 += 64) {
          const double bv = s_beta[min(c0 + lane, kn - 1)];
          const int cn = min(64, kn - c0);
          for (int j = 0; j < cn; ++j) {
            prod *= lane_f64(bv, j);
            E += prod;
          }
        }
        if (lane == 0) {
          lds[7] = static_cast<uint64_t>(__double_as_longlong(prod));
          lds[6] = static_cast<uint64_t>(__double_as_longlong(E));
          if (k0 + kn == K) a.exp_len[b] = static_cast<float>(E);
        }
      }
      __syncthreads();
    }
  }
  if (a.trajectory) return;
  __syncthreads();
  const int ks = s_ks;
  const bool residual = ks < k_.K;
  int tok = -1;
  if (residual || a.Kp == k_.K + 1) {
    const int64_t V = k_.V;
    const int nT = k_.nT;
    const int R = static_cast<int>(k_.R);
    const float* prow = a.logp + (b * a.Kp + ks) * V;
    const int64_t m0 = (b * k_.K + (residual ? ks : 0)) * k_.R;
    const uint32_t r = draw(k_.seed, kResidual, static_cast<uint32_t>(ks),
                            static_cast<uint64_t>(k_.seq_offset + b), k_.step);
    // The tile from the residual's tile sums, or from the target's when the residual has no
    // mass (and for the bonus row).
    Pick pk{-1, 0, 0};
    if (residual)
      pk = pick_block(nT, [&](int t) { return a.res_tiles[b * nT + t]; }, weigh_u64, r, lds);
    const bool use_res = pk.i >= 0;
    if (!use_res)
      pk = pick_block(nT, [&](int t) { return a.p_tiles[b * nT + t]; }, weigh_u64, r, lds);
    if (pk.i >= 0) {
      // The tile's integer weights into LDS, with one round of loads by the whole workgroup:
      // P(v), and for the residual the branch values detexp32(lq_z(v)) of every category.
      const int64_t v0 = static_cast<int64_t>(pk.i) * kTile;
      const int n = static_cast<int>(V - v0 < kTile ? V - v0 : kTile);
      const float pv = prow[v0 + min(tid, n - 1)];  // raw values first, clamped indices
      const double wv = a.wpost[m0 + min(tid, R - 1)];
      auto stage = [&](int base) {  // kStageBatch branch values per thread, loads first
        float lq[kStageBatch];
#pragma unroll
        for (int j = 0; j < kStageBatch; ++j) {  // clamped indices: every load is in bounds
          const int idx = min(base + tid + 256 * j, R * kTile - 1);
          const int64_t m = m0 + idx / kTile;
          const int i = min(idx & (kTile - 1), n - 1);
          lq[j] = flat_lq(k_.tls[m * V + v0 + i], k_.lmass[m * nT + pk.i], k_.lse[m]);
        }
#pragma unroll
        for (int j = 0; j < kStageBatch; ++j) {
          const int idx = base + tid + 256 * j;
          if (idx < R * kTile) s_y[idx] = detexp32(lq[j]);
        }
      };
      if (use_res) {
        stage(0);  // R <= 16: straight-line, in flight with the two loads above
        for (int base = kStageBatch * 256; base < R * kTile; base += kStageBatch * 256)
          stage(base);
      }
      if (tid < n) s_wt[tid] = quant_detexp32(pv);
      if (use_res && tid < R) wz[tid] = wv;
      __syncthreads();
      if (use_res && tid < n) {
        // R(v) = max(P(v) - Q(v), 0), Q(v) = floor((sum over ascending z of
        // w_z detexp32(lq_z(v))) 2^40): the weights the residual's tile sums were taken from.
        double Q = 0.0;
        for (int z = 0; z < R; ++z)
          Q = __dadd_rn(Q, __dmul_rn(wz[z], static_cast<double>(s_y[z * kTile + tid])));
        const uint64_t P = s_wt[tid], Qi = quant40d(Q);
        s_wt[tid] = P > Qi ? P - Qi : 0;
      }
      __syncthreads();
      tok = pick_in_tile(s_wt, n, pk, lds);
    }
  }
  if (tid == 0) a.next_token[b] = tok;
}

__global__ __launch_bounds__(256) void finalize_kernel(VerifyArgs a, int nchunk) {
  finalize_block(a, blockIdx.x, nchunk);
}

// The acceptance-mass stream with the residual tile sums folded in (V % 4 == 0, masses
// requested). Workgroup g handles chunk c = g % nchunk (stream_tiles(R) vocabulary tiles: 40, or
// 32 at R <= 4, where cpw consecutive chunks share a workgroup) of position row k of block b,
// g / nchunk = k B + b:
//  * k < K: the R branch rows and the target row of the chunk are read once for the
//    acceptance-mass partial; at the block's first rejected position the same loaded values also
//    give the contract's integer residual and target tile sums (weights as in residual_body), so
//    no row is read twice;
//  * k = K (rows of the bonus row, present when Kp = K + 1): read only when the block accepted
//    every position, for the bonus row's integer tile sums.
// The finalize launch that follows reduces the partials and draws. Finalising in the last of a
// block's workgroups to finish instead (a per-block arrival counter after device-coherent
// partial stores) measured slower: every workgroup held its slot through the store
// acknowledgement and the counter's round trip (Qwen3-8B verification call 0.2339 ms with the
// separate launch against 0.2504 ms).
constexpr float kLog2eChunk = 1.4426950408889634f;

// Eight waves per SIMD (64 VGPRs) up to eight categories: the binary64 residual arithmetic, which
// only the workgroups at a first rejection run, would otherwise set the register budget of every
// workgroup. Sixteen categories keep their 16 row loads in flight in 80 VGPRs (six waves).
template <int RT>
constexpr int stream_waves() { return RT > 8 ? 6 : 8; }

// Chunks per workgroup: a chunk streams (R + 1) x 16 KB per position row, so at R <= 4 several
// chunks share a workgroup's start-up when the grid stays large (stress shape, R = 4: 1.157 ->
// 1.088 ms with four, 1.009 with eight, 1.008 with sixteen, 1.230 with all 37 in one); at R = 8
// a chunk loop measured 6% slower even at one chunk, so R > 4 keeps one chunk per workgroup
// and no loop.
constexpr int kStreamChunksSmallR = 8;
constexpr int64_t kStreamMinGroups = 2048;  // one workgroup per slot at eight waves per SIMD
__host__ __device__ constexpr bool stream_multi_chunk(int rt) { return rt > 0 && rt <= 4; }

// Vocabulary tiles per stream chunk: 32 where several chunks share a workgroup, else 40 (30
// chunks per row at V = 151,936: fewer, longer workgroups whose count fills whole rounds of the
// 2048 slots at the Qwen3 shapes: verification call 0.2257 -> 0.2226 ms at Qwen3-8B and
// 0.1221 -> 0.1201 ms at Qwen3-4B; 48 tiles measured 0.2235 and 0.1233).
__host__ __device__ constexpr int stream_tiles(int rt) { return stream_multi_chunk(rt) ? 32 : 40; }
// The workspace holds n_chunks(nT) partials per position (kTilesPerChunk-tile chunks): no stream
// chunk may be narrower, or the stream would write past them.
static_assert(stream_tiles(0) >= kTilesPerChunk && stream_tiles(1) >= kTilesPerChunk,
              "stream chunks narrower than the workspace's");

template <int RT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(stream_waves<RT>(), 8)))
void verify_stream_kernel(VerifyArgs a, int nchunk, int cpw) {
  constexpr int TPC = stream_tiles(RT);  // vocabulary tiles per chunk
  const int CPW = stream_multi_chunk(RT) ? cpw : 1;
  const BlockArgs& k_ = a.blk;
  const int64_t B = k_.B;
  const int ncw = (nchunk + CPW - 1) / CPW;
  const int cw = static_cast<int>(blockIdx.x % static_cast<unsigned>(ncw));
  const int64_t pb = blockIdx.x / static_cast<unsigned>(ncw);
  const int64_t k = pb / B, b = pb % B;
  const int R = RT > 0 ? RT : static_cast<int>(k_.R);
  const int64_t V = k_.V;
  const int tid = threadIdx.x;
  __shared__ float s_w[kMaxR];
  __shared__ double s_wz[kMaxR];
  __shared__ float s_offx[kMaxR][TPC];  // fl32(lmass - lse) of the chunk's tiles
  __shared__ float red[4];
  const int ks = a.trajectory ? -1 : a.n_accept[b];  // first rejected position, K if none
  const bool bonus = k == k_.K;
  const bool res = !a.trajectory && (bonus ? ks == k_.K : k == ks);
  const int64_t m0 = (b * k_.K + k) * k_.R;  // first branch row of the position (k < K)
#pragma unroll 1
  for (int cc = 0; cc < CPW; ++cc) {
  const int c = cw * CPW + cc;
  if (c >= nchunk) break;       // workgroup-uniform
  if (cc > 0) __syncthreads();  // the previous chunk's readers of s_offx and red are done
  const int t0 = c * TPC;
  const int nt = min(TPC, k_.nT - t0);
  if (!bonus) {
    for (int i = tid; i < R * TPC; i += blockDim.x) {
      const int z = i / TPC, tt = i % TPC;
      if (tt < nt) s_offx[z][tt] = k_.lmass[(m0 + z) * k_.nT + t0 + tt] - k_.lse[m0 + z];
    }
    if (cc == 0 && tid < R) {
      const double wv = a.wpost[m0 + tid];
      s_w[tid] = static_cast<float>(wv);
      s_wz[tid] = wv;
    }
  }
  __syncthreads();
  const int64_t vb = static_cast<int64_t>(t0) * kTile;
  const int64_t ve = min(V, vb + static_cast<int64_t>(nt) * kTile);
  const float* prow = a.logp + (b * a.Kp + k) * V;
  const float* trow = k_.tls + m0 * V;
  float acc = 0.0f;
  if (!bonus || res) {
#pragma unroll 1
    for (int i = 0; i < TPC * kTile / 1024; ++i) {
      const int64_t v = vb + 4 * tid + 1024 * i;
      const int tt = (4 * tid + 1024 * i) >> 7;  // the 32 threads of a half-wave share a tile
      uint64_t sp = 0, sr = 0;
      if (v < ve) {
        const float4 p = load_stream4(prow + v);
        if (!bonus && !res) {
          float q0 = 0.0f, q1 = 0.0f, q2 = 0.0f, q3 = 0.0f;
          if constexpr (RT > 0) {
            float4 x[RT];
#pragma unroll
            for (int z = 0; z < RT; ++z) x[z] = load_stream4(trow + z * V + v);
#pragma unroll
            for (int z = 0; z < RT; ++z) {
              const float o = s_offx[z][tt] * kLog2eChunk, w = s_w[z];
              q0 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(x[z].x, kLog2eChunk, o)), q0);
              q1 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(x[z].y, kLog2eChunk, o)), q1);
              q2 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(x[z].z, kLog2eChunk, o)), q2);
              q3 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(x[z].w, kLog2eChunk, o)), q3);
            }
          } else {
            for (int z = 0; z < R; ++z) {
              const float4 xz = load_stream4(trow + z * V + v);
              const float o = s_offx[z][tt] * kLog2eChunk, w = s_w[z];
              q0 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(xz.x, kLog2eChunk, o)), q0);
              q1 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(xz.y, kLog2eChunk, o)), q1);
              q2 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(xz.z, kLog2eChunk, o)), q2);
              q3 = fmaf(w, __builtin_amdgcn_exp2f(fmaf(xz.w, kLog2eChunk, o)), q3);
            }
          }
          acc += fminf(__builtin_amdgcn_exp2f(p.x * kLog2eChunk), q0) +
                 fminf(__builtin_amdgcn_exp2f(p.y * kLog2eChunk), q1) +
                 fminf(__builtin_amdgcn_exp2f(p.z * kLog2eChunk), q2) +
                 fminf(__builtin_amdgcn_exp2f(p.w * kLog2eChunk), q3);
        } else if (!bonus) {
          // The first rejected position: one pass over each branch row feeds both the binary32
          // mixture of the acceptance mass (same operations in the same order as above) and the
          // contract's binary64 mixture of the residual weights, so no row is read twice (with
          // every wave of the chip streaming, a second read would miss the L2).
          const float pe[4] = {p.x, p.y, p.z, p.w};
          float q[4] = {0.0f, 0.0f, 0.0f, 0.0f};
          double Q[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 1
          for (int z = 0; z < R; ++z) {
            const float4 xz = load_stream4(trow + z * V + v);
            const float xe[4] = {xz.x, xz.y, xz.z, xz.w};
            const float oz = s_offx[z][tt];
            const float o = oz * kLog2eChunk, w = s_w[z];
            const double wz = s_wz[z];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              q[e] = fmaf(w, __builtin_amdgcn_exp2f(fmaf(xe[e], kLog2eChunk, o)), q[e]);
              Q[e] = __dadd_rn(Q[e], __dmul_rn(wz, static_cast<double>(detexp32(__fadd_rn(xe[e], oz)))));
            }
          }
          acc += fminf(__builtin_amdgcn_exp2f(p.x * kLog2eChunk), q[0]) +
                 fminf(__builtin_amdgcn_exp2f(p.y * kLog2eChunk), q[1]) +
                 fminf(__builtin_amdgcn_exp2f(p.z * kLog2eChunk), q[2]) +
                 fminf(__builtin_amdgcn_exp2f(p.w * kLog2eChunk), q[3]);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint64_t P = quant_detexp32(pe[e]);
            const uint64_t Qi = quant40d(Q[e]);
            sr += P > Qi ? P - Qi : 0;
            sp += P;
          }
        } else {  // the bonus row after full acceptance: P only
          sp = (quant_detexp32(p.x) + quant_detexp32(p.y)) +
               (quant_detexp32(p.z) + quant_detexp32(p.w));
        }
      }
      if (res) {  // workgroup-uniform: every lane of the half-wave takes part
#pragma unroll
        for (int o = 16; o > 0; o >>= 1) {
          sp += __shfl_xor(sp, o);
          sr += __shfl_xor(sr, o);
        }
        if ((tid & 31) == 0 && tt < nt) {
          a.p_tiles[b * k_.nT + t0 + tt] = sp;
          if (!bonus) a.res_tiles[b * k_.nT + t0 + tt] = sr;
        }
      }
    }
  }
  if (!bonus) {
    acc = wave_sum_f32(acc);
    if ((tid & 63) == 0) red[tid >> 6] = acc;
    __syncthreads();
    if (tid == 0)
      a.beta_part[(b * k_.K + k) * nchunk + c] = (red[0] + red[1]) + (red[2] + red[3]);
  }
  }
}

}  // namespace

hipError_t launch_verify(const VerifyArgs& a, hipStream_t stream) {
  const int64_t B = a.blk.B;
  const int64_t npos = B * a.blk.K;
  const int nchunk = n_chunks(a.blk.nT);
  if (npos > 0x7fffffff) return hipErrorInvalidConfiguration;
  if (a.blk.K * a.blk.R <= kChainMaxKR && a.blk.K <= kChainMaxK)
    hipLaunchKernelGGL(chain_parallel_kernel, dim3(static_cast<unsigned>(B)), dim3(256), 0, stream,
                       a);
  else
    hipLaunchKernelGGL(chain_kernel, dim3(static_cast<unsigned>(B)), dim3(64), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const bool want_beta = a.beta || a.exp_len;
  const bool stream_path = want_beta && (a.blk.V & 3) == 0 && !a.trajectory;
  int nchunk_f = nchunk;  // the finalisation's partials per position
  if (stream_path) {
    // One stream: acceptance masses, and the residual tile sums at the first rejection from the
    // same loads. Trajectory mode keeps the beta kernel below: its stream has no residual
    // arithmetic to carry, and at R = 16 it measured 3.48 ms against 3.78 ms fused per 128-block
    // chunk.
    const int rows = static_cast<int>(a.blk.K) + (!a.trajectory && a.Kp == a.blk.K + 1 ? 1 : 0);
    const int64_t R = a.blk.R;  // the template argument of the launch below: R, or 0
    const int rt = R == 1 || R == 2 || R == 4 || R == 8 || R == 16 ? static_cast<int>(R) : 0;
    const int nchunk_s = (a.blk.nT + stream_tiles(rt) - 1) / stream_tiles(rt);
    nchunk_f = nchunk_s;
    const int64_t cw_many = (nchunk_s + kStreamChunksSmallR - 1) / kStreamChunksSmallR;
    const int cpw = stream_multi_chunk(rt) && rows * B * cw_many >= kStreamMinGroups
                        ? kStreamChunksSmallR : 1;
    const int64_t nwg = static_cast<int64_t>(rows) * B * ((nchunk_s + cpw - 1) / cpw);
    if (nwg > 0x7fffffff) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<unsigned>(nwg));
    switch (a.blk.R) {
      case 1: hipLaunchKernelGGL(verify_stream_kernel<1>, grid, dim3(256), 0, stream, a, nchunk_s, cpw); break;
      case 2: hipLaunchKernelGGL(verify_stream_kernel<2>, grid, dim3(256), 0, stream, a, nchunk_s, cpw); break;
      case 4: hipLaunchKernelGGL(verify_stream_kernel<4>, grid, dim3(256), 0, stream, a, nchunk_s, cpw); break;
      case 8: hipLaunchKernelGGL(verify_stream_kernel<8>, grid, dim3(256), 0, stream, a, nchunk_s, cpw); break;
      case 16: hipLaunchKernelGGL(verify_stream_kernel<16>, grid, dim3(256), 0, stream, a, nchunk_s, cpw); break;
      default: hipLaunchKernelGGL(verify_stream_kernel<0>, grid, dim3(256), 0, stream, a, nchunk_s, cpw); break;
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  } else if (want_beta && !a.trajectory) {
    if (npos + B > 0x7fffffff) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<unsigned>(B + npos), nchunk);
    switch (a.blk.R) {
      case 1: hipLaunchKernelGGL(beta_residual_kernel<1>, grid, dim3(256), 0, stream, a); break;
      case 2: hipLaunchKernelGGL(beta_residual_kernel<2>, grid, dim3(256), 0, stream, a); break;
      case 4: hipLaunchKernelGGL(beta_residual_kernel<4>, grid, dim3(256), 0, stream, a); break;
      case 8: hipLaunchKernelGGL(beta_residual_kernel<8>, grid, dim3(256), 0, stream, a); break;
      case 16: hipLaunchKernelGGL(beta_residual_kernel<16>, grid, dim3(256), 0, stream, a); break;
      default: hipLaunchKernelGGL(beta_residual_kernel<0>, grid, dim3(256), 0, stream, a); break;
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  } else if (want_beta) {
    const dim3 grid(static_cast<unsigned>(npos), nchunk);
    switch (a.blk.R) {
      case 1: hipLaunchKernelGGL(beta_kernel<1>, grid, dim3(256), 0, stream, a); break;
      case 2: hipLaunchKernelGGL(beta_kernel<2>, grid, dim3(256), 0, stream, a); break;
      case 4: hipLaunchKernelGGL(beta_kernel<4>, grid, dim3(256), 0, stream, a); break;
      case 8: hipLaunchKernelGGL(beta_kernel<8>, grid, dim3(256), 0, stream, a); break;
      case 16: hipLaunchKernelGGL(beta_kernel<16>, grid, dim3(256), 0, stream, a); break;
      default: hipLaunchKernelGGL(beta_kernel<0>, grid, dim3(256), 0, stream, a); break;
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  } else if (!a.trajectory) {
    const dim3 grid(static_cast<unsigned>(B), nchunk);
    switch (a.blk.R) {
      case 1: hipLaunchKernelGGL(residual_kernel<1>, grid, dim3(256), 0, stream, a); break;
      case 2: hipLaunchKernelGGL(residual_kernel<2>, grid, dim3(256), 0, stream, a); break;
      case 4: hipLaunchKernelGGL(residual_kernel<4>, grid, dim3(256), 0, stream, a); break;
      case 8: hipLaunchKernelGGL(residual_kernel<8>, grid, dim3(256), 0, stream, a); break;
      case 16: hipLaunchKernelGGL(residual_kernel<16>, grid, dim3(256), 0, stream, a); break;
      default: hipLaunchKernelGGL(residual_kernel<0>, grid, dim3(256), 0, stream, a); break;
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (want_beta || !a.trajectory) {
    hipLaunchKernelGGL(finalize_kernel, dim3(static_cast<unsigned>(B)), dim3(256), 0, stream, a,
                       nchunk_f);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace dbl
