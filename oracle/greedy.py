"""Greedy-branch proposal: block draw and stochastic verification. CPU oracle.

TEST INFRASTRUCTURE (see ``oracle/contract.py``): only tests, the smoke check and the benchmark's
CPU baseline use this module; the GPU library never does.

The paper's reported experiments draw a category from the (temperature-scaled) prior and then
decode that branch greedily (Sec. "Drafter sampling during inference"; appendix
"Greedy-Branch Proposal"). With x_hat[k, z] = argmax_v q_k(v | y, z) the branch tokens
(lowest index on ties), the proposal is the finite mixture of deterministic blocks

    q_greedy(x_1..x_K) = sum_z pi_z prod_k 1{x_k = x_hat[k, z]}        (Eq. greedy-branch-proposal)

with pi = softmax(l / Z_T) (Z_T = 0: the highest-prior category). Verification uses the
prefix-marginalised conditional of the same mixture (appendix "Prefix-Marginalized
Conditional"): the consistent set C_k = {z : x_hat[j, z] = x_j for all j < k}, the weights
pi~_{k,z} = pi_z 1{z in C_k} / sum_{z' in C_k} pi_z', and

    q_greedy(v | x_<k) = sum_{z in C_k} pi~_{k,z} 1{v = x_hat[k, z]}  (Eq. appendix-greedy-conditional)

a distribution supported on at most R tokens. Acceptance, the residual max(p - q, 0) and the
bonus token follow Algorithm "Greedy-Branch Dependent Speculative Verification" exactly as in the
soft case (appendix "Distributional Correctness").

Determinism contract (as ``oracle/mixture.py``): pi~ is the log-domain normalisation of
L_z = log prior (l_z / Z_T) restricted to C_k (-inf outside), with the deterministic binary64
exponential and an ascending-z sum; q at a token is the binary64 sum over ascending z of the
matching weights; probabilities that decide are quantised to 2^-40; draws are the Philox words of
``oracle/contract.py`` with the same purposes as the soft mode (category 0, accept 2, residual or
bonus 3; no token draws: the branch is decoded greedily). beta, AL_b and E are real-valued outputs
in ordinary binary64 arithmetic.
"""
from __future__ import annotations

import numpy as np

from .contract import (PURPOSE_ACCEPT, PURPOSE_CATEGORY, PURPOSE_RESIDUAL, accept_int,
                       detexp32, icdf, quant40)
from .mixture import draws, normalize_weights, prior, prior_log_weights


def branch_tokens(logits):
    """x_hat = argmax over the last axis (the vocabulary), lowest index on ties."""
    return np.argmax(np.asarray(logits), axis=-1).astype(np.int32)


def sample_blocks_greedy(xhat, ell, z_temp, seed, step, seq):
    """z ~ pi^(Z_T) (inverse CDF on the quantised prior, Philox purpose 0) and x = x_hat[:, z].

    xhat [B, K, R] int branch tokens, ell [B, R] float32, seq [B]. Returns z [B], x [B, K]
    (int32; a block whose prior has no quantised mass gets z = -1 and x = -1).
    """
    xhat = np.asarray(xhat, dtype=np.int64)
    B, K, R = xhat.shape
    seq = np.asarray(seq)
    pi_q = quant40(prior(ell, z_temp))
    r_cat = draws(seed, PURPOSE_CATEGORY, 0, seq, step)
    z = np.array([icdf(pi_q[b], r_cat[b]) for b in range(B)], dtype=np.int32)
    x = np.full((B, K), -1, dtype=np.int32)
    for b in range(B):
        if z[b] >= 0:
            x[b] = xhat[b, :, z[b]]
    return z, x


def _conditional_weights(L0, consistent):
    """pi~ over the consistent set: log-domain normalisation of L0 restricted to it."""
    return normalize_weights(np.where(consistent, L0, -np.inf))


def _q_at(w, xhat_k, v):
    """q_greedy(v | prefix) = sum over ascending z of w_z 1{x_hat[k, z] = v}, binary64.
    w [B, R], xhat_k [B, R], v [B]."""
    Q = np.zeros(w.shape[0])
    for z in range(w.shape[1]):
        Q = Q + w[:, z] * (xhat_k[:, z] == v).astype(np.float64)
    return Q


def _support(w_b, xhat_kb):
    """{token: q_greedy(token)} for one block and position; tokens in first-seen z order."""
    out = {}
    for z in range(len(w_b)):
        if w_b[z] > 0:
            t = int(xhat_kb[z])
            out[t] = out.get(t, 0.0) + float(w_b[z])
    return out


def _beta_greedy(w, xhat_k, logp_k):
    """beta = sum_v min(p(v), q_greedy(v)) over the (at most R) support tokens, binary64."""
    B = w.shape[0]
    beta = np.zeros(B)
    for b in range(B):
        for t, qv in _support(w[b], xhat_k[b]).items():
            if 0 <= t < logp_k.shape[-1]:
                beta[b] += min(float(np.exp(np.float64(logp_k[b, t]))), qv)
    return beta


def _prefix_sum_of_products(a):
    return np.sum(np.cumprod(np.asarray(a, dtype=np.float64), axis=-1), axis=-1)


def verify_blocks_greedy(xhat, ell, z_temp, x, logp, seed, step, seq, with_beta=True):
    """Sequential verification of drafted blocks against the greedy-branch conditional.

    xhat [B, K, R] branch tokens, ell [B, R], x [B, K] drafted tokens (ids outside [0, V) have
    zero target probability), logp [B, Kp, V] with Kp in {K, K + 1}. Returns a dict with
    n_accept [B], next_token [B] (-1 when all K are accepted and no bonus row is given),
    q [B, K] = q_greedy(x_k | x_<k), A [B, K], al [B], w [B, K, R] the weights pi~, and,
    when ``with_beta``, beta [B, K] and E [B].
    """
    xhat = np.asarray(xhat, dtype=np.int64)
    logp = np.asarray(logp, dtype=np.float32)
    x = np.asarray(x, dtype=np.int64)
    B, K, R = xhat.shape
    Kp, V = logp.shape[1], logp.shape[2]
    if Kp not in (K, K + 1):
        raise ValueError("logp must hold K or K + 1 rows per block")
    seq = np.asarray(seq)
    bi = np.arange(B)
    L0 = prior_log_weights(ell, z_temp)
    consistent = np.ones((B, R), dtype=bool)
    W = np.empty((B, K, R))
    Qk = np.empty((B, K))
    A = np.empty((B, K))
    beta = np.empty((B, K))
    n_accept = np.zeros(B, dtype=np.int32)
    alive = np.ones(B, dtype=bool)
    for k in range(K):
        w = _conditional_weights(L0, consistent)
        W[:, k] = w
        xk = x[:, k]
        ok = (xk >= 0) & (xk < V)
        Qx = _q_at(w, xhat[:, k], xk)
        Px = np.where(ok, detexp32(logp[bi, k, np.clip(xk, 0, V - 1)]), np.float32(0))
        Px = Px.astype(np.float64)
        Qk[:, k] = Qx
        with np.errstate(divide="ignore", invalid="ignore"):
            A[:, k] = np.where(Qx > 0, np.minimum(1.0, Px / np.where(Qx > 0, Qx, 1.0)),
                               np.where(Px > 0, 1.0, 0.0))
        r_acc = draws(seed, PURPOSE_ACCEPT, k, seq, step)
        q_i, p_i = quant40(Qx), quant40(Px)
        for b in range(B):
            if alive[b]:
                if accept_int(r_acc[b], q_i[b], p_i[b]):
                    n_accept[b] += 1
                else:
                    alive[b] = False
        if with_beta:
            beta[:, k] = _beta_greedy(w, xhat[:, k], logp[:, k])
        consistent &= xhat[:, k, :] == xk[:, None]

    next_token = np.full(B, -1, dtype=np.int32)
    for b in range(B):
        ks = int(n_accept[b])
        if ks < K:
            p_int = quant40(detexp32(logp[b, ks]))
            q_int = np.zeros(V, dtype=np.uint64)
            for t, qv in _support(W[b, ks], xhat[b, ks]).items():
                if 0 <= t < V:
                    q_int[t] = quant40(np.float64(qv))
            res = np.where(p_int > q_int, p_int - q_int, np.uint64(0)).astype(np.uint64)
            r = draws(seed, PURPOSE_RESIDUAL, ks, seq[b:b + 1], step)[0]
            tok = icdf(res, r)
            if tok < 0:
                tok = icdf(p_int, r)
            next_token[b] = tok
        elif Kp == K + 1:
            r = draws(seed, PURPOSE_RESIDUAL, K, seq[b:b + 1], step)[0]
            next_token[b] = icdf(quant40(detexp32(logp[b, K])), r)

    out = dict(n_accept=n_accept, next_token=next_token, q=Qk, A=A, w=W,
               al=_prefix_sum_of_products(A))
    if with_beta:
        out["beta"] = beta
        out["E"] = _prefix_sum_of_products(beta)
    return out


def expected_len_greedy(xhat, ell, z_temp, xs, logp):
    """beta_k = sum_v min(p_k(v), q_greedy(v | xs_<k)) along a given trajectory xs and
    E = sum_i prod_{j<=i} beta_j. Returns (beta [B, K], E [B]) in binary64."""
    xhat = np.asarray(xhat, dtype=np.int64)
    logp = np.asarray(logp, dtype=np.float32)
    xs = np.asarray(xs, dtype=np.int64)
    B, K, R = xhat.shape
    L0 = prior_log_weights(ell, z_temp)
    consistent = np.ones((B, R), dtype=bool)
    beta = np.empty((B, K))
    for k in range(K):
        w = _conditional_weights(L0, consistent)
        beta[:, k] = _beta_greedy(w, xhat[:, k], logp[:, k])
        consistent &= xhat[:, k, :] == xs[:, k, None]
    return beta, _prefix_sum_of_products(beta)
