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
//   finalize  one wavefront per block: acceptance masses, E = sum_i prod_{j<=i} beta_j, and the
//             residual/bonus inverse-CDF draw.
// The same kernels serve the expected-length reduction along a given trajectory (no accept
// test, no residual). Built with floating-point contraction off (determinism contract).
#include <hip/hip_runtime.h>
#include <stdint.h>

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
    for (int z = 0; z < R; ++z) Q = __dadd_rn(Q, __dmul_rn(__shfl(w, z), __shfl(y, z)));
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

// Acceptance-mass stream. Thread i of the workgroup handles 4 consecutive ids per step.
__global__ __launch_bounds__(256) void beta_kernel(VerifyArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t pos = blockIdx.x;
  const int64_t b = pos / k_.K;
  const int64_t k = pos % k_.K;
  const int R = static_cast<int>(k_.R);
  __shared__ float wz[kMaxR];
  __shared__ float red[4];
  if (threadIdx.x < R) wz[threadIdx.x] = static_cast<float>(a.wpost[pos * k_.R + threadIdx.x]);
  __syncthreads();
  const int64_t v_begin = static_cast<int64_t>(blockIdx.y) * kTilesPerChunk * kTile;
  const int64_t v_end = min(k_.V, v_begin + static_cast<int64_t>(kTilesPerChunk) * kTile);
  const float* prow = a.logp + (b * a.Kp + k) * k_.V;
  const int64_t m0 = pos * k_.R;
  float acc = 0.0f;
  for (int64_t v = v_begin + 4 * threadIdx.x; v < v_end; v += 4 * blockDim.x) {
    const int n = static_cast<int>(min<int64_t>(4, v_end - v));
    float p[4], q[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      p[e] = e < n ? __expf(prow[v + e]) : 0.0f;
      q[e] = 0.0f;
    }
    const int t = static_cast<int>(v / kTile);
    for (int z = 0; z < R; ++z) {
      const int64_t m = m0 + z;
      const float off = k_.lmass[m * k_.nT + t] - k_.lse[m];
      const float* row = k_.tls + m * k_.V;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (e < n) q[e] += wz[z] * __expf(row[v + e] + off);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) acc += fminf(p[e], q[e]);
  }
  acc = wave_sum_f32(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0)
    a.beta_part[pos * gridDim.y + blockIdx.y] = (red[0] + red[1]) + (red[2] + red[3]);
}

// Integer weight of id v in the residual / bonus distributions.
struct ResidualWeight {
  const float* tls;
  const float* lmass;
  const float* lse;
  const float* prow;   // target row at the position
  int64_t m0;          // first branch row of the position
  int64_t V;
  int nT, R;
  const double* w;     // posterior at the position (R values)
  __device__ uint64_t p_int(int64_t v) const { return quant40(detexp32(prow[v])); }
  __device__ uint64_t q_int(int64_t v) const {
    double Q = 0.0;
    for (int z = 0; z < R; ++z) {
      const int64_t m = m0 + z;
      const float lq = flat_lq(tls[m * V + v], lmass[m * nT + v / kTile], lse[m]);
      Q = __dadd_rn(Q, __dmul_rn(w[z], static_cast<double>(detexp32(lq))));
    }
    return quant40d(Q);
  }
  __device__ uint64_t res_int(int64_t v) const {
    const uint64_t P = p_int(v), Q = q_int(v);
    return P > Q ? P - Q : 0;
  }
};

__global__ __launch_bounds__(256) void residual_kernel(VerifyArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t b = blockIdx.x;
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int ks = a.n_accept[b];
  const bool residual = ks < k_.K;
  if (!residual && a.Kp != k_.K + 1) return;
  __shared__ double wz[kMaxR];
  if (residual && threadIdx.x < k_.R)
    wz[threadIdx.x] = a.wpost[(b * k_.K + ks) * k_.R + threadIdx.x];
  __syncthreads();
  ResidualWeight W{k_.tls, k_.lmass, k_.lse, a.logp + (b * a.Kp + ks) * k_.V,
                   (b * k_.K + (residual ? ks : 0)) * k_.R, k_.V, k_.nT,
                   static_cast<int>(k_.R), wz};
  const int t_begin = blockIdx.y * kTilesPerChunk;
  const int t_end = min(k_.nT, t_begin + kTilesPerChunk);
  for (int t = t_begin + wave; t < t_end; t += 4) {
    uint64_t sp = 0, sr = 0;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int64_t v = static_cast<int64_t>(t) * kTile + 2 * lane + e;
      if (v < k_.V) {
        const uint64_t P = W.p_int(v);
        sp += P;
        if (residual) {
          const uint64_t Q = W.q_int(v);
          sr += P > Q ? P - Q : 0;
        }
      }
    }
    sp = wave_sum_u64(sp);
    sr = wave_sum_u64(sr);
    if (lane == 0) {
      a.p_tiles[b * k_.nT + t] = sp;
      a.res_tiles[b * k_.nT + t] = sr;
    }
  }
}

__global__ __launch_bounds__(64) void finalize_kernel(VerifyArgs a, int nchunk) {
  const BlockArgs& k_ = a.blk;
  const int64_t b = blockIdx.x;
  const int lane = lane_id();
  if (a.beta || a.exp_len) {
    double prod = 1.0, E = 0.0;
    for (int64_t k = 0; k < k_.K; ++k) {
      const float* part = a.beta_part + (b * k_.K + k) * nchunk;
      double s = 0.0;
      for (int c = lane; c < nchunk; c += 64) s += static_cast<double>(part[c]);
      s = wave_sum_f64(s);
      if (a.beta && lane == 0) a.beta[b * k_.K + k] = static_cast<float>(s);
      prod *= s;
      E += prod;
    }
    if (a.exp_len && lane == 0) a.exp_len[b] = static_cast<float>(E);
  }
  if (a.trajectory) return;
  const int ks = a.n_accept[b];
  const bool residual = ks < k_.K;
  int tok = -1;
  if (residual || a.Kp == k_.K + 1) {
    __shared__ double wz[kMaxR];
    if (residual && lane < k_.R) wz[lane] = a.wpost[(b * k_.K + ks) * k_.R + lane];
    __syncthreads();
    ResidualWeight W{k_.tls, k_.lmass, k_.lse, a.logp + (b * a.Kp + ks) * k_.V,
                     (b * k_.K + (residual ? ks : 0)) * k_.R, k_.V, k_.nT,
                     static_cast<int>(k_.R), wz};
    const uint32_t r = draw(k_.seed, kResidual, static_cast<uint32_t>(ks),
                            static_cast<uint64_t>(k_.seq_offset + b), k_.step);
    if (residual)
      tok = select_by_tiles(a.res_tiles + b * k_.nT, k_.nT, k_.V, r,
                            [&](int64_t v) { return W.res_int(v); });
    if (tok < 0)
      tok = select_by_tiles(a.p_tiles + b * k_.nT, k_.nT, k_.V, r,
                            [&](int64_t v) { return W.p_int(v); });
  }
  if (lane == 0) a.next_token[b] = tok;
}

}  // namespace

hipError_t launch_verify(const VerifyArgs& a, hipStream_t stream) {
  const int64_t B = a.blk.B;
  const int64_t npos = B * a.blk.K;
  const int nchunk = n_chunks(a.blk.nT);
  if (npos > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(chain_kernel, dim3(static_cast<unsigned>(B)), dim3(64), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const bool want_beta = a.beta || a.exp_len;
  if (want_beta) {
    hipLaunchKernelGGL(beta_kernel, dim3(static_cast<unsigned>(npos), nchunk), dim3(256), 0,
                       stream, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (!a.trajectory) {
    hipLaunchKernelGGL(residual_kernel, dim3(static_cast<unsigned>(B), nchunk), dim3(256), 0,
                       stream, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (want_beta || !a.trajectory) {
    hipLaunchKernelGGL(finalize_kernel, dim3(static_cast<unsigned>(B)), dim3(64), 0, stream, a,
                       nchunk);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace dbl
