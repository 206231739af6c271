// Greedy-branch mode (appendix "Greedy-Branch Proposal", "Prefix-Marginalized Conditional",
// Algorithm "Greedy-Branch Dependent Speculative Verification"): a category is drawn from the
// prior and its branch is decoded greedily, x_k = x_hat[k, z] = argmax_v q_k(v | z). The
// proposal conditional at position k is supported on at most R tokens:
//     q(v | x_<k) = sum_{z in C_k} pi~_{k,z} 1{v = x_hat[k, z]},
// C_k = {z : x_hat[j, z] = x_j for j < k}, pi~ = the prior renormalised over C_k. No vocabulary
// row of the drafter is read: the draw and the verifier take only the branch tokens.
//   greedy_sample    one wavefront per block: category draw, branch copy;
//   greedy_chain     one wavefront per block, lane = category: consistent set, pi~ (log-domain
//                    normalisation of the prior restricted to C_k), q at the drafted token, the
//                    accept chain, A_k / AL_b, beta_k over the support tokens and E; for staged
//                    blocks (the usual case) a parallel form handles every position at once;
//   greedy_ptiles    grid (block, vocabulary chunk): integer tile sums of the target row at the
//                    first rejected position (or the bonus row);
//   greedy_finalize  one 256-thread workgroup per block: the residual tile sums are the target
//                    tile sums minus min(P, Q) at the support tokens; inverse-CDF draw.
// Built with floating-point contraction off (determinism contract).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "contract.hpp"
#include "kernels.hpp"
#include "wave.hpp"

namespace dbl {
namespace {

__device__ __forceinline__ bool in_vocab(int32_t x, int64_t V) { return x >= 0 && x < V; }

__global__ __launch_bounds__(64) void greedy_sample_kernel(GreedyArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t b = blockIdx.x;
  const int lane = lane_id();
  const int z = draw_category(k_, b);
  if (lane == 0) a.z_out[b] = z;
  for (int64_t k = lane; k < k_.K; k += 64)
    a.x_out[b * k_.K + k] = z >= 0 ? a.xhat[(b * k_.K + k) * k_.R + z] : -1;
}

// Positions per block whose inputs the chain stages in LDS before walking them (drafted token,
// branch tokens and the target log-probabilities at both): the walk then waits on no memory.
constexpr int kGreedyStageK = 64;
constexpr int kGreedyStageKR = 1024;

__global__ __launch_bounds__(64) void greedy_chain_kernel(GreedyArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t b = blockIdx.x;
  const int lane = lane_id();
  const int R = static_cast<int>(k_.R);
  const int64_t V = k_.V;
  const uint64_t seq = static_cast<uint64_t>(k_.seq_offset + b);
  __shared__ int32_t s_tok[64];
  __shared__ double s_w[64];
  __shared__ int32_t s_x[kGreedyStageK];
  __shared__ float s_px[kGreedyStageK];
  __shared__ int32_t s_t[kGreedyStageKR];
  __shared__ float s_pt[kGreedyStageKR];
  const bool staged = k_.K <= kGreedyStageK && k_.K * k_.R <= kGreedyStageKR;
  if (staged) {  // every gather of the walk, issued together
    const int K = static_cast<int>(k_.K), KR = K * R;
    for (int k = lane; k < K; k += 64) s_x[k] = a.x[b * k_.K + k];
    for (int i = lane; i < KR; i += 64) s_t[i] = a.xhat[b * k_.K * k_.R + i];
    __syncthreads();
    for (int k = lane; k < K; k += 64) {
      const int32_t xk = s_x[k];
      s_px[k] = in_vocab(xk, V) ? a.logp[(b * a.Kp + k) * V + xk] : 0.0f;
    }
    for (int i = lane; i < KR; i += 64) {
      const int32_t t = s_t[i];
      s_pt[i] = in_vocab(t, V) ? a.logp[(b * a.Kp + i / R) * V + t] : 0.0f;
    }
    __syncthreads();
  }
  const double L0 = prior_log_weight(k_.prior + b * k_.R, R, k_.z_temp);
  const bool want_beta = a.beta || a.exp_len;
  bool consistent = lane < R;
  bool alive = true;
  int n_acc = 0;
  double prodA = 1.0, al = 0.0, prodB = 1.0, E = 0.0;
  for (int64_t k = 0; k < k_.K; ++k) {
    const int64_t row = (b * k_.K + k) * k_.R;
    const double w = normalize_weight(consistent ? L0 : -INFINITY, R);
    if (lane < R) a.wpost[row + lane] = w;
    const int32_t xk = staged ? s_x[k] : a.x[b * k_.K + k];
    const int32_t t = lane < R ? (staged ? s_t[k * R + lane] : a.xhat[row + lane]) : -1;
    const bool match = lane < R && t == xk;
    const float* prow = a.logp + (b * a.Kp + k) * V;
    if (!a.trajectory) {
      double Q = 0.0;
      for (int z = 0; z < R; ++z) Q = __dadd_rn(Q, lane_f64(match ? w : 0.0, z));
      const float px = staged ? s_px[k] : (in_vocab(xk, V) ? prow[xk] : 0.0f);
      const double P = in_vocab(xk, V) ? static_cast<double>(detexp32(px)) : 0.0;
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
    if (want_beta) {
      s_tok[lane] = t;
      s_w[lane] = lane < R ? w : 0.0;
      __syncthreads();
      // Lane z represents its token if it is the lowest category with weight on that token;
      // q(token) is the ascending-z sum of the weights of every category proposing it.
      double contrib = 0.0;
      if (lane < R && w > 0.0 && in_vocab(t, V)) {
        bool first = true;
        double q = 0.0;
        for (int z = 0; z < R; ++z) {
          if (s_w[z] > 0.0 && s_tok[z] == t) {
            if (z < lane) first = false;
            q = __dadd_rn(q, s_w[z]);
          }
        }
        const float pt = staged ? s_pt[k * R + lane] : prow[t];
        if (first) contrib = fmin(exp(static_cast<double>(pt)), q);
      }
      const double beta_k = wave_sum_f64(contrib);
      if (a.beta && lane == 0) a.beta[b * k_.K + k] = static_cast<float>(beta_k);
      prodB *= beta_k;
      E += prodB;
      __syncthreads();
    }
    consistent = consistent && match;
  }
  if (lane == 0) {
    if (!a.trajectory) {
      a.n_accept[b] = n_acc;
      if (a.al) a.al[b] = static_cast<float>(al);
    }
    if (a.exp_len) a.exp_len[b] = static_cast<float>(E);
  }
}

// Parallel form of greedy_chain_kernel for staged blocks (K <= kGreedyStageK and
// K * R <= kGreedyStageKR), one 256-thread workgroup per block. The consistent set at position k
// depends only on the drafted prefix, so every position is handled at once: lane z of the
// wavefront holding position k reads whether branch z matched every drafted token before k (a
// bit mask per branch), normalises pi~ with the same wavefront operations, and forms q at the
// drafted token and beta_k over the support tokens; one thread then takes E in position order,
// and wavefront 0 runs the integer accept chain. Bit-identical to greedy_chain_kernel.
__global__ __launch_bounds__(256) void greedy_chain_parallel_kernel(GreedyArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid >> 6;
  constexpr int kWaves = 4;
  const int R = static_cast<int>(k_.R);
  const int K = static_cast<int>(k_.K);
  const int KR = K * R;
  const int64_t V = k_.V;
  const uint64_t seq = static_cast<uint64_t>(k_.seq_offset + b);
  __shared__ int32_t s_x[kGreedyStageK];
  __shared__ float s_px[kGreedyStageK];
  __shared__ int32_t s_t[kGreedyStageKR];
  __shared__ float s_pt[kGreedyStageKR];
  __shared__ double s_L0[kMaxR];
  __shared__ uint64_t s_mask[kMaxR];  // bit k: branch z's token is the drafted token at k
  __shared__ double s_w[kWaves][64];
  __shared__ double s_Q[kGreedyStageK];
  __shared__ double s_P[kGreedyStageK];
  __shared__ double s_beta[kGreedyStageK];
  for (int k = tid; k < K; k += blockDim.x) s_x[k] = a.x[b * k_.K + k];
  for (int i = tid; i < KR; i += blockDim.x) s_t[i] = a.xhat[b * k_.K * k_.R + i];
  if (wave == 0) {
    const double l0 = prior_log_weight(k_.prior + b * k_.R, R, k_.z_temp);
    if (lane < R) s_L0[lane] = l0;
  }
  __syncthreads();
  for (int k = tid; k < K; k += blockDim.x) {
    const int32_t xk = s_x[k];
    s_px[k] = in_vocab(xk, V) ? a.logp[(b * a.Kp + k) * V + xk] : 0.0f;
  }
  for (int i = tid; i < KR; i += blockDim.x) {
    const int32_t t = s_t[i];
    s_pt[i] = in_vocab(t, V) ? a.logp[(b * a.Kp + i / R) * V + t] : 0.0f;
  }
  if (tid < R) {
    uint64_t m = 0;
    for (int k = 0; k < K; ++k)
      if (s_t[k * R + tid] == s_x[k]) m |= uint64_t{1} << k;
    s_mask[tid] = m;
  }
  __syncthreads();
  const bool want_beta = a.beta || a.exp_len;
  for (int k = wave; k < K; k += kWaves) {
    const uint64_t before = (uint64_t{1} << k) - 1;  // positions 0 .. k - 1 (k < 64)
    const bool consistent = lane < R && (s_mask[lane] & before) == before;
    const double w = normalize_weight(consistent ? s_L0[lane] : -INFINITY, R);
    const int64_t row = (b * k_.K + k) * k_.R;
    if (lane < R) a.wpost[row + lane] = w;
    const int32_t xk = s_x[k];
    const int32_t t = lane < R ? s_t[k * R + lane] : -1;
    const bool match = lane < R && t == xk;
    if (!a.trajectory) {
      double Q = 0.0;
      for (int z = 0; z < R; ++z) Q = __dadd_rn(Q, lane_f64(match ? w : 0.0, z));
      const double P = in_vocab(xk, V) ? static_cast<double>(detexp32(s_px[k])) : 0.0;
      if (lane == 0) {
        s_Q[k] = Q;
        s_P[k] = P;
      }
    }
    if (want_beta) {
      s_w[wave][lane] = lane < R ? w : 0.0;
      // Wavefront-private LDS: the writes above precede these reads in the wavefront's queue.
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // Lane z represents its token if it is the lowest category with weight on that token;
      // q(token) is the ascending-z sum of the weights of every category proposing it.
      double contrib = 0.0;
      if (lane < R && w > 0.0 && in_vocab(t, V)) {
        bool first = true;
        double q = 0.0;
        for (int z = 0; z < R; ++z) {
          if (s_w[wave][z] > 0.0 && s_t[k * R + z] == t) {
            if (z < lane) first = false;
            q = __dadd_rn(q, s_w[wave][z]);
          }
        }
        if (first) contrib = fmin(exp(static_cast<double>(s_pt[k * R + lane])), q);
      }
      const double beta_k = wave_sum_f64(contrib);
      if (lane == 0) {
        s_beta[k] = beta_k;
        if (a.beta) a.beta[b * k_.K + k] = static_cast<float>(beta_k);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
  }
  __syncthreads();
  if (tid == 0 && a.exp_len) {
    double prodB = 1.0, E = 0.0;
    for (int k = 0; k < K; ++k) {
      prodB *= s_beta[k];
      E += prodB;
    }
    a.exp_len[b] = static_cast<float>(E);
  }
  if (a.trajectory || wave != 0) return;
  // Wavefront 0: every position's accept test at once (the draws do not depend on earlier
  // outcomes); n_accept is the first rejection, and the running product of the A_k is taken in
  // position order by every lane alike.
  const int k = lane;
  bool rej = false;
  double A = 0.0;
  if (k < K) {
    const double Q = s_Q[k], P = s_P[k];
    A = Q > 0.0 ? fmin(1.0, P / Q) : (P > 0.0 ? 1.0 : 0.0);
    const uint32_t r = draw(k_.seed, kAccept, static_cast<uint32_t>(k), seq, k_.step);
    rej = !accept_int(r, quant40d(Q), quant40d(P));
  }
  const uint64_t rejm = __ballot(rej);
  const int n_acc = rejm ? __ffsll(static_cast<unsigned long long>(rejm)) - 1 : K;
  double prodA = 1.0, al = 0.0;
  for (int j = 0; j < K; ++j) {
    prodA = __dmul_rn(prodA, lane_f64(A, j));
    al = __dadd_rn(al, prodA);
  }
  if (lane == 0) {
    a.n_accept[b] = n_acc;
    if (a.al) a.al[b] = static_cast<float>(al);
  }
}

// Integer tile sums floor(detexp32(logp) 2^40) of the target row at position n_accept[b] (the
// first rejected position, or the bonus row K); 8 lanes per 128-id tile.
__global__ __launch_bounds__(256) void greedy_ptiles_kernel(GreedyArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t b = blockIdx.x;
  const int ks = a.n_accept[b];
  if (ks >= k_.K && a.Kp != k_.K + 1) return;
  const int sub = threadIdx.x & 7;
  const int t = blockIdx.y * kTilesPerChunk + (threadIdx.x >> 3);
  const int64_t V = k_.V;
  uint64_t sp = 0;
  if (t < k_.nT) {
    const int64_t v0 = static_cast<int64_t>(t) * kTile;
    const float* prow = a.logp + (b * a.Kp + ks) * V + v0;
    if ((V & 3) == 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int v = 4 * sub + 32 * i;
        if (v0 + v < V) {
          const float4 p4 = load_stream4(prow + v);
          sp += quant_detexp32(p4.x) + quant_detexp32(p4.y) + quant_detexp32(p4.z) +
                quant_detexp32(p4.w);
        }
      }
    } else {
      for (int i = 0; i < 16; ++i) {
        const int v = sub + 8 * i;
        if (v0 + v < V) sp += quant_detexp32(prow[v]);
      }
    }
  }
  sp += __shfl_xor(sp, 1);
  sp += __shfl_xor(sp, 2);
  sp += __shfl_xor(sp, 4);
  if (sub == 0 && t < k_.nT) a.p_tiles[b * k_.nT + t] = sp;
}

__global__ __launch_bounds__(256) void greedy_finalize_kernel(GreedyArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t b = blockIdx.x;
  const int tid = threadIdx.x;
  const int64_t V = k_.V;
  const int nT = k_.nT;
  __shared__ uint64_t lds[8];
  __shared__ int32_t s_tok[kMaxR];
  __shared__ uint64_t s_q[kMaxR];
  __shared__ double s_qd[kMaxR];
  __shared__ double s_wz[kMaxR];
  __shared__ int32_t s_tz[kMaxR];
  __shared__ uint64_t s_p[kMaxR];
  __shared__ int s_n;
  const int ks = a.n_accept[b];
  const bool residual = ks < k_.K;
  if (!residual && a.Kp != k_.K + 1) {
    if (tid == 0) a.next_token[b] = -1;
    return;
  }
  const float* prow = a.logp + (b * a.Kp + ks) * V;
  const uint32_t r = draw(k_.seed, kResidual, static_cast<uint32_t>(ks),
                          static_cast<uint64_t>(k_.seq_offset + b), k_.step);
  auto p_int = [&](int64_t v) { return quant_detexp32(prow[v]); };
  int tok = -1;
  if (residual) {
    // The posterior and branch tokens at ks, gathered in parallel.
    const int64_t row = (b * k_.K + ks) * k_.R;
    if (tid < k_.R) {
      s_wz[tid] = a.wpost[row + tid];
      s_tz[tid] = a.xhat[row + tid];
    }
    __syncthreads();
    if (tid == 0) {
      // Support of q at ks: distinct branch tokens of the categories with weight, with
      // q(token) summed over ascending z and quantised.
      int n = 0;
      for (int z = 0; z < k_.R; ++z) {
        const double w = s_wz[z];
        if (!(w > 0.0)) continue;
        const int32_t t = s_tz[z];
        int j = 0;
        while (j < n && s_tok[j] != t) ++j;
        if (j == n) {
          s_tok[n] = t;
          s_qd[n++] = 0.0;
        }
        s_qd[j] = __dadd_rn(s_qd[j], w);
      }
      for (int j = 0; j < n; ++j) s_q[j] = quant40d(s_qd[j]);
      s_n = n;
    }
    for (int t = tid; t < nT; t += blockDim.x)
      a.res_tiles[b * nT + t] = a.p_tiles[b * nT + t];
    __syncthreads();
    if (tid < s_n && in_vocab(s_tok[tid], V)) s_p[tid] = p_int(s_tok[tid]);
    __syncthreads();
    if (tid == 0) {
      for (int j = 0; j < s_n; ++j) {
        if (!in_vocab(s_tok[j], V)) continue;
        const uint64_t P = s_p[j];
        a.res_tiles[b * nT + s_tok[j] / kTile] -= P < s_q[j] ? P : s_q[j];
      }
    }
    __syncthreads();
    const int n = s_n;
    tok = select_by_tiles_block(
        a.res_tiles + b * nT, nT, V, r,
        [&](int64_t v) {
          const uint64_t P = p_int(v);
          uint64_t Q = 0;
          for (int j = 0; j < n; ++j)
            if (s_tok[j] == v) Q = s_q[j];
          return P > Q ? P - Q : 0;
        },
        lds);
  }
  if (tok < 0) tok = select_by_tiles_block(a.p_tiles + b * nT, nT, V, r, p_int, lds);
  if (tid == 0) a.next_token[b] = tok;
}

}  // namespace

hipError_t launch_sample_greedy(const GreedyArgs& a, hipStream_t stream) {
  if (a.blk.B > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(greedy_sample_kernel, dim3(static_cast<unsigned>(a.blk.B)), dim3(64), 0,
                     stream, a);
  return hipGetLastError();
}

hipError_t launch_verify_greedy(const GreedyArgs& a, hipStream_t stream) {
  const int64_t B = a.blk.B;
  if (B > 0x7fffffff) return hipErrorInvalidConfiguration;
  if (a.blk.K <= kGreedyStageK && a.blk.K * a.blk.R <= kGreedyStageKR)
    hipLaunchKernelGGL(greedy_chain_parallel_kernel, dim3(static_cast<unsigned>(B)), dim3(256), 0,
                       stream, a);
  else
    hipLaunchKernelGGL(greedy_chain_kernel, dim3(static_cast<unsigned>(B)), dim3(64), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.trajectory) return e;
  hipLaunchKernelGGL(greedy_ptiles_kernel, dim3(static_cast<unsigned>(B), n_chunks(a.blk.nT)),
                     dim3(256), 0, stream, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(greedy_finalize_kernel, dim3(static_cast<unsigned>(B)), dim3(256), 0, stream,
                     a);
  return hipGetLastError();
}

}  // namespace dbl
