// Forward quantities of the acceptance-oriented training surrogate (Sec. "Acceptance-Oriented
// Training") along target trajectories x*: prefix log-likelihoods of the dependent proposal
// log q(x*_{1:l}) = log sum_z pi_z prod_{j<=l} q_j(x*_j | z) (Eq. cp-drafter) and of the target,
// the importance ratios log r_l (Eq. acceptance-length-objective), the acceptance probabilities
// A_j = min(1, p_j(x*_j) / q(x*_j | x*_<j)) with the conditional as a ratio of consecutive
// prefix likelihoods, S_l = sum_{i<=l} prod_{j<=i} A_j, the truncation l_tau and the per-block
// surrogate J = sum_{l<=l_tau} (log r_l + log S_l) (Eq. subblock-objective), and the marginalised
// block NLL -log q(x*_{1:K}) (Eq. dependent-nll).
//
// One wavefront per block, lane = category: each lane accumulates its branch's log-likelihood of
// the trajectory prefix in binary64 and the wavefront takes the log-sum-exp over categories at
// every prefix length. Only K * R gathered branch log-probabilities and K target log-probabilities
// are read per block.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "contract.hpp"
#include "kernels.hpp"
#include "wave.hpp"

namespace dbl {
namespace {

__device__ __forceinline__ double wave_logsumexp(double v) {
  const double m = wave_max_f64(v);
  if (!(m > -INFINITY)) return -INFINITY;
  return m + log(wave_sum_f64(exp(v - m)));
}

__global__ __launch_bounds__(64) void objective_kernel(ObjectiveArgs a) {
  const BlockArgs& k_ = a.blk;
  const int64_t b = blockIdx.x;
  const int lane = lane_id();
  const int R = static_cast<int>(k_.R);
  const int64_t V = k_.V;
  // log pi_z: the prior's log-weights normalised over the categories.
  const double L0 = prior_log_weight(k_.prior + b * k_.R, R, k_.z_temp);
  const double lse0 = wave_logsumexp(lane < R ? L0 : -INFINITY);  // whole wavefront active
  const double log_pi = lane < R ? L0 - lse0 : -INFINITY;
  const double log_tau = log(static_cast<double>(a.tau));
  double cum = log_pi, prev_logq = 0.0, logp_cum = 0.0, prodA = 1.0, S = 0.0, J = 0.0;
  double logq = 0.0;
  int ell_tau = static_cast<int>(k_.K);
  bool done = false;
  for (int64_t j = 0; j < k_.K; ++j) {
    const int32_t x = a.x[b * k_.K + j];
    const bool ok = x >= 0 && x < V;
    const int64_t row = (b * k_.K + j) * k_.R + lane;
    const float lq = ok && lane < R
                         ? flat_lq(k_.tls[row * V + x], k_.lmass[row * k_.nT + x / kTile], k_.lse[row])
                         : -INFINITY;
    cum += static_cast<double>(lq);
    logq = wave_logsumexp(lane < R ? cum : -INFINITY);
    const double lp = ok ? static_cast<double>(a.logp[(b * k_.K + j) * V + x]) : -INFINITY;
    logp_cum += lp;
    const double A = fmin(1.0, exp(lp - (logq - prev_logq)));
    prodA *= A;
    S += prodA;
    const double log_r = logq - logp_cum;
    if (!done) {
      J += log_r + log(S);
      if (log_r < log_tau) {
        done = true;
        ell_tau = static_cast<int>(j) + 1;
      }
    }
    if (lane == 0) {
      if (a.log_r) a.log_r[b * k_.K + j] = static_cast<float>(log_r);
      if (a.S) a.S[b * k_.K + j] = static_cast<float>(S);
    }
    prev_logq = logq;
  }
  if (lane == 0) {
    a.ell_tau[b] = ell_tau;
    a.J[b] = static_cast<float>(J);
    a.nll[b] = static_cast<float>(-logq);
  }
}

}  // namespace

hipError_t launch_objective(const ObjectiveArgs& a, hipStream_t stream) {
  if (a.blk.B > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(objective_kernel, dim3(static_cast<unsigned>(a.blk.B)), dim3(64), 0, stream,
                     a);
  return hipGetLastError();
}

}  // namespace dbl
