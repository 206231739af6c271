"""Training-objective forward quantities on target trajectories: CPU oracle.

TEST INFRASTRUCTURE (see ``oracle/contract.py``): only tests, the smoke check and the benchmark's
CPU baseline use this module; the GPU library never does.

For a target-generated block x*_{1:K} (Sec. "Acceptance-Oriented Training"; the paper's b is K
here and its K is R) and the dependent proposal of Eq. cp-drafter with prior pi = softmax(l / Z_T):

* prefix log-likelihoods  log q(x*_{1:l}) = log sum_z pi_z prod_{j<=l} q_j(x*_j | z)  and
  log p(x*_{1:l}) = sum_{j<=l} log p_j(x*_j)  (products of the gathered per-token target
  probabilities, "Target probabilities during training");
* the marginalised block negative log-likelihood  NLL = -log q(x*_{1:K})  (Eq. dependent-nll;
  with R = 1 it is Eq. independent-nll);
* the importance ratio  log r_l = log q(x*_{1:l}) - log p(x*_{1:l})  of Eq.
  acceptance-length-objective;
* the acceptance probabilities  A_j = min(1, p_j(x*_j) / q(x*_j | x*_<j))  with the
  prefix-marginalised conditional q(x_j | x_<j) = q(x_{1:j}) / q(x_{1:j-1}), and
  S_l = sum_{i<=l} prod_{j<=i} A_j;
* the truncation  l_tau = min({l : r_l < tau} U {K})  and the per-block surrogate
  J = sum_{l=1}^{l_tau} (log r_l + log S_l)  (Eq. subblock-objective; the training loss is
  -J averaged over trajectories, Eq. training-loss). The paper uses tau = 0.1.

Everything is binary64 computed from the binary32 branch log-probabilities and target
log-probabilities (no quantisation: these are real-valued outputs; l_tau is an integer decided by
a binary64 comparison).
"""
from __future__ import annotations

import numpy as np

from .mixture import prior


def _logsumexp(a, axis=-1):
    a = np.asarray(a, dtype=np.float64)
    m = np.max(a, axis=axis, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    with np.errstate(divide="ignore"):
        return np.squeeze(m, axis) + np.log(np.sum(np.exp(a - m), axis=axis))


def acceptance_objective(lq, ell, z_temp, xs, logp, tau=0.1):
    """Per-block objective quantities along trajectories xs.

    lq [B, K, R, V] float32 branch log-probabilities, ell [B, R], xs [B, K] target trajectory,
    logp [B, K, V] float32 target log-probabilities. Returns a dict with log_q [B, K] =
    log q(x*_{1:l}), log_p [B, K], log_r [B, K], A [B, K], S [B, K], ell_tau [B] (1-based),
    J [B] and nll [B].
    """
    lq = np.asarray(lq, dtype=np.float32)
    logp = np.asarray(logp, dtype=np.float32)
    xs = np.asarray(xs, dtype=np.int64)
    B, K, R, V = lq.shape
    bi = np.arange(B)
    with np.errstate(divide="ignore"):
        log_pi = np.log(prior(ell, z_temp))                          # [B, R]
    # log prod_{j<=l} q_j(x*_j | z) for every l, then the mixture over z
    lq_x = np.stack([lq[bi, j, :, xs[:, j]] for j in range(K)], axis=1).astype(np.float64)
    branch = log_pi[:, None, :] + np.cumsum(lq_x, axis=1)          # [B, K, R]
    log_q = _logsumexp(branch, axis=-1)                             # [B, K]
    lp_x = np.stack([logp[bi, j, xs[:, j]] for j in range(K)], axis=1).astype(np.float64)
    log_p = np.cumsum(lp_x, axis=1)
    log_r = log_q - log_p
    prev = np.concatenate([np.zeros((B, 1)), log_q[:, :-1]], axis=1)
    with np.errstate(over="ignore", invalid="ignore"):
        A = np.minimum(1.0, np.exp(lp_x - (log_q - prev)))
    S = np.cumsum(np.cumprod(A, axis=1), axis=1)
    below = log_r < np.log(tau)
    ell_tau = np.where(below.any(axis=1), np.argmax(below, axis=1) + 1, K).astype(np.int32)
    J = np.empty(B)
    with np.errstate(divide="ignore"):
        terms = log_r + np.log(S)
    for b in range(B):
        J[b] = np.sum(terms[b, :ell_tau[b]])
    return dict(log_q=log_q, log_p=log_p, log_r=log_r, A=A, S=S, ell_tau=ell_tau, J=J,
                nll=-log_q[:, -1])
