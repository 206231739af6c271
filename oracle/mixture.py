"""Latent-mixture block proposal, block draw and stochastic verification: CPU oracle.

TEST INFRASTRUCTURE (see ``oracle/contract.py``).

Notation. A batch holds B independent blocks. Each block has K drafted positions k = 0..K-1 and
R latent categories z (the paper writes b for the block length and K for the number of
categories). For block b the inputs are

* lq[b, k, z, :]  binary32 log q_k(. | y, z), the branch token log-probabilities;
* for the draw, the same log-probabilities in the head's two-level form: tls[b, k, z, :]
  (log-probability within each 128-id tile), lmass[b, k, z, :] (tile log-masses) and
  lse[b, k, z] (their log-sum-exp), lq = fl32(tls + fl32(lmass - lse));
* ell[b, :]       binary32 category logits l_z(y);
* logp[b, k, :]   binary32 target log-probabilities p_k(.) = p(. | y, x_<k); an optional extra
                  row k = K feeds the bonus token.

What is computed, in the paper's order:

1. Category prior with temperature Z_T (Sec. "Drafter sampling during inference"):
   q_{Z_T}(z) = softmax(l / Z_T); Z_T = 0 selects the highest-prior category (appendix,
   "Greedy-Branch Proposal"), ties going to the lowest index.
2. Block draw from the mixture of Eq. cp-drafter: first z ~ q_{Z_T}, then every position
   independently from q_k(. | z). The paper leaves open how a token is drawn from q_k(. | z);
   here it is drawn in two stages that follow the two-level form: first the 128-id tile t
   with probability exp(lmass_t - lse), then the id v within it with probability exp(tls_v)
   (their product is q_k(v | z)), each stage an inverse CDF on its quantised weights.
3. Verification of a drafted block with the prefix-marginalised conditional of
   Eq. dep-conditional, computed through the category posterior of Eq. category-posterior,
       w_{k,z} proportional to q_{Z_T}(z) prod_{j<k} q_j(x_j | z),
   and the next-token mixture of Eq. dep-next-token-distribution,
       q_k(v | x_<k) = sum_z w_{k,z} q_k(v | z).
   Position k is accepted with probability min(1, p_k(x_k) / q_k(x_k | x_<k)) (Eq. accept-prob)
   while every earlier position was accepted; at the first rejection a replacement is drawn
   from the normalised positive residual max(p_k - q_k, 0) and verification stops; if every
   position was accepted and the target row for position K is supplied, a bonus token is
   drawn from it (Algorithm "Greedy-Branch Dependent Speculative Verification", last step).
4. Quantities that describe acceptance:
   A_k = min(1, p_k(x_k) / q_k(x_k | x_<k)) and AL_b(x) = sum_i prod_{j<=i} A_j
   (Eq. acceptance-length); the acceptance mass beta_k = sum_v min(p_k(v), q_k(v | x_<k)),
   the probability that position k is accepted given the prefix (a single position gives
   1 - TV(p, q)); and E = sum_i prod_{j<=i} beta_j along the conditioning prefix (the draft,
   or a given target trajectory for ``expected_len_blocks``).

Discrete decisions follow the determinism contract of ``oracle/contract.py``: the posterior
is normalised in the log domain with the deterministic binary64 exponential and an
ascending-z sum; token probabilities that feed a decision use the deterministic binary32
exponential; the mixture at a token is the binary64 sum over ascending z of w_z * q_z; all
sampled distributions are quantised to 2^-40. beta, AL_b and E are real-valued outputs and use
ordinary binary64 arithmetic.
"""
from __future__ import annotations

import numpy as np

from .contract import (PURPOSE_ACCEPT, PURPOSE_CATEGORY, PURPOSE_RESIDUAL, PURPOSE_TOKEN,
                       accept_int, detexp32, dexp64, icdf, philox4x32_10_np, quant40)


def draws(seed: int, purpose: int, k: int, seq, step: int, word: int = 0):
    """Philox word ``word`` (0 or 1) for (purpose, k) and every sequence index in ``seq``."""
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    seq = np.asarray(seq, dtype=np.uint64)
    out = philox4x32_10_np(k, purpose, seq, int(step), seed & 0xFFFFFFFF, seed >> 32)
    return out[word]


# ----------------------------------------------------------------------------------------
# 1. Category prior and posterior
# ----------------------------------------------------------------------------------------
def prior_log_weights(ell, z_temp: float):
    """Unnormalised log prior L_z: l_z / Z_T when Z_T > 0; when Z_T = 0, 0 at the argmax, -inf elsewhere."""
    ell = np.asarray(ell, dtype=np.float32)
    if z_temp < 0:
        raise ValueError("category temperature must be >= 0")
    if z_temp > 0:
        return ell.astype(np.float64) / np.float64(np.float32(z_temp))
    top = np.argmax(ell, axis=-1)        # first index of the maximum
    L = np.full(ell.shape, -np.inf)
    np.put_along_axis(L, top[..., None], 0.0, axis=-1)
    return L


def normalize_weights(L):
    """w_z = exp(L_z - max_z L) / sum_z exp(L_z - max_z L) over the last axis.

    The exponential is the deterministic binary64 one, the sum runs over ascending z and the
    division is one correctly rounded binary64 division. A row whose maximum is -inf (an
    impossible prefix) gets all-zero weights.
    """
    L = np.asarray(L, dtype=np.float64)
    mx = np.max(L, axis=-1, keepdims=True)
    dead = ~np.isfinite(mx)
    e = dexp64(np.where(dead, -np.inf, L - np.where(dead, 0.0, mx)))
    S = np.zeros(L.shape[:-1])
    for z in range(L.shape[-1]):
        S = S + e[..., z]
    with np.errstate(invalid="ignore", divide="ignore"):
        w = e / S[..., None]
    return np.where(dead, 0.0, w)


def prior(ell, z_temp: float):
    """q_{Z_T}(z | y) for every block, binary64 [B, R]."""
    return normalize_weights(prior_log_weights(ell, z_temp))


def _mixture_fp64(w, y):
    """sum_z w[..., z] * y[..., z, :] in binary64, z ascending; w [..., R], y [..., R, V]."""
    Q = np.zeros(y.shape[:-2] + y.shape[-1:])
    for z in range(y.shape[-2]):
        Q = Q + w[..., z, None] * y[..., z, :].astype(np.float64)
    return Q


# ----------------------------------------------------------------------------------------
# 2. Block draw
# ----------------------------------------------------------------------------------------
TILE = 128  # ids per tile of the two-level form


def draw_token(tls_row, lmass_row, lse, r_tile: int, r_id: int) -> int:
    """One token from the two-level form of a branch row: the tile by an inverse CDF on
    floor(detexp32(fl32(lmass_t - lse)) 2^40) with word r_tile, then the id within it by an
    inverse CDF on floor(detexp32(tls_v) 2^40) with word r_id. -1 if no tile has quantised
    mass."""
    tls_row = np.asarray(tls_row, dtype=np.float32)
    lmass_row = np.asarray(lmass_row, dtype=np.float32)
    off = (lmass_row - np.float32(lse)).astype(np.float32)
    t = icdf(quant40(detexp32(off)), r_tile)
    if t < 0:
        return -1
    ids = tls_row[t * TILE:(t + 1) * TILE]
    j = icdf(quant40(detexp32(ids)), r_id)
    return -1 if j < 0 else t * TILE + j


def sample_blocks(tls, lmass, lse, ell, z_temp, seed, step, seq):
    """Draw z ~ q_{Z_T} and x_k ~ q_k(. | z) for every block.

    tls [B, K, R, V], lmass [B, K, R, nT], lse [B, K, R] float32 (the two-level form of the
    branch log-probabilities), ell [B, R] float32, seq [B] global sequence indices.
    Returns z [B] int32 and x [B, K] int32 (-1 marks a row with no quantised mass).
    """
    tls = np.asarray(tls, dtype=np.float32)
    lmass = np.asarray(lmass, dtype=np.float32)
    lse = np.asarray(lse, dtype=np.float32)
    B, K, R, V = tls.shape
    seq = np.asarray(seq)
    pi_q = quant40(prior(ell, z_temp))
    r_cat = draws(seed, PURPOSE_CATEGORY, 0, seq, step)
    z = np.array([icdf(pi_q[b], r_cat[b]) for b in range(B)], dtype=np.int32)
    x = np.empty((B, K), dtype=np.int32)
    for k in range(K):
        r_tile = draws(seed, PURPOSE_TOKEN, k, seq, step, word=0)
        r_id = draws(seed, PURPOSE_TOKEN, k, seq, step, word=1)
        for b in range(B):
            zb = z[b]
            x[b, k] = draw_token(tls[b, k, zb], lmass[b, k, zb], lse[b, k, zb], r_tile[b],
                                 r_id[b])
    return z, x


# ----------------------------------------------------------------------------------------
# 3-4. Verification, acceptance mass and expected length
# ----------------------------------------------------------------------------------------
def _beta(w, lq_k, logp_k):
    """beta = sum_v min(p(v), sum_z w_z q_z(v)) in binary64; w [B, R], lq_k [B, R, V]."""
    p = np.exp(np.asarray(logp_k, dtype=np.float64))
    q = np.zeros_like(p)
    for z in range(lq_k.shape[1]):
        q = q + w[:, z, None] * np.exp(lq_k[:, z, :].astype(np.float64))
    return np.sum(np.minimum(p, q), axis=-1)


def _prefix_sum_of_products(a):
    """sum_i prod_{j<=i} a_j along the last axis, binary64."""
    a = np.asarray(a, dtype=np.float64)
    return np.sum(np.cumprod(a, axis=-1), axis=-1)


def verify_blocks(lq, ell, z_temp, x, logp, seed, step, seq, with_beta=True):
    """Sequential stochastic verification of drafted blocks.

    lq [B, K, R, V], ell [B, R], x [B, K] drafted tokens, logp [B, Kp, V] with Kp in {K, K+1}.
    Returns a dict with n_accept [B], next_token [B] (-1 when all K are accepted and no bonus
    row is given), A [B, K], al [B] = AL_b(x), w [B, K, R] posterior weights, and, when
    ``with_beta``, beta [B, K] and E [B].
    """
    lq = np.asarray(lq, dtype=np.float32)
    logp = np.asarray(logp, dtype=np.float32)
    x = np.asarray(x, dtype=np.int64)
    B, K, R, V = lq.shape
    Kp = logp.shape[1]
    if Kp not in (K, K + 1):
        raise ValueError("logp must hold K or K + 1 rows per block")
    seq = np.asarray(seq)
    bi = np.arange(B)

    L = prior_log_weights(ell, z_temp)
    W = np.empty((B, K, R))
    A = np.empty((B, K))
    beta = np.empty((B, K))
    n_accept = np.zeros(B, dtype=np.int32)
    alive = np.ones(B, dtype=bool)
    for k in range(K):
        w = normalize_weights(L)
        W[:, k] = w
        lq_x = lq[bi, k, :, x[:, k]]                      # [B, R] log q_k(x_k | z)
        y = detexp32(lq_x)
        Qx = np.zeros(B)
        for z in range(R):
            Qx = Qx + w[:, z] * y[:, z].astype(np.float64)
        Px = detexp32(logp[bi, k, x[:, k]]).astype(np.float64)
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
            beta[:, k] = _beta(w, lq[:, k], logp[:, k])
        L = L + lq_x.astype(np.float64)

    next_token = np.full(B, -1, dtype=np.int32)
    for b in range(B):
        ks = int(n_accept[b])
        if ks < K:
            Y = detexp32(lq[b, ks])                       # [R, V]
            Q = _mixture_fp64(W[b, ks], Y)
            q_int = quant40(Q)
            p_int = quant40(detexp32(logp[b, ks]))
            res = np.where(p_int > q_int, p_int - q_int, np.uint64(0)).astype(np.uint64)
            r = draws(seed, PURPOSE_RESIDUAL, ks, seq[b:b + 1], step)[0]
            tok = icdf(res, r)
            if tok < 0:
                tok = icdf(p_int, r)
            next_token[b] = tok
        elif Kp == K + 1:
            r = draws(seed, PURPOSE_RESIDUAL, K, seq[b:b + 1], step)[0]
            next_token[b] = icdf(quant40(detexp32(logp[b, K])), r)

    out = dict(n_accept=n_accept, next_token=next_token, A=A, w=W,
               al=_prefix_sum_of_products(A))
    if with_beta:
        out["beta"] = beta
        out["E"] = _prefix_sum_of_products(beta)
    return out


def expected_len_blocks(lq, ell, z_temp, xs, logp):
    """beta_k along a given trajectory xs and E = sum_i prod_{j<=i} beta_j.

    lq [B, K, R, V], ell [B, R], xs [B, K] conditioning trajectory (e.g. drawn from the
    target), logp [B, K, V]. Returns (beta [B, K], E [B]) in binary64.
    """
    lq = np.asarray(lq, dtype=np.float32)
    logp = np.asarray(logp, dtype=np.float32)
    xs = np.asarray(xs, dtype=np.int64)
    B, K, R, V = lq.shape
    bi = np.arange(B)
    L = prior_log_weights(ell, z_temp)
    beta = np.empty((B, K))
    for k in range(K):
        w = normalize_weights(L)
        beta[:, k] = _beta(w, lq[:, k], logp[:, k])
        L = L + lq[bi, k, :, xs[:, k]].astype(np.float64)
    return beta, _prefix_sum_of_products(beta)
