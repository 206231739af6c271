"""Drafter output head of DBLast: CPU oracle.

TEST INFRASTRUCTURE (see ``oracle/contract.py``).

Sec. "Architecture": every category branch h_{i,z} is mapped by the shared target LM head to
token logits, and q_i(. | y, z) is their softmax. Here the head is the plain definition, in
binary64, on the exact input values (binary32 or bfloat16 values held in binary32 arrays):

    logits[m, v] = sum_j h[m, j] * w[v, j]          (w is the [V, d] lm_head.weight layout)
    logq[m, v]   = logits[m, v] - log sum_u exp(logits[m, u])

Row m of h is block position (b, k) and category r, m = (b * K + k) * R + r.

The library hands log-probabilities over in a two-level form that one pass over V can write:
for vocabulary tile t (columns [128 t, 128 t + 128) clipped to V)

    lmass[m, t] = log sum_{v in t} exp(logits[m, v])     (log-mass of the tile)
    tls[m, v]   = logits[m, v] - lmass[m, t(v)]          (log-prob of v within its tile)
    lse[m]      = log sum_v exp(logits[m, v])

so that logq = tls + (lmass - lse). ``flat_logq`` rebuilds the binary32 log-probability that
every consumer uses: fl32(tls + fl32(lmass - lse)).
"""
from __future__ import annotations

import numpy as np

VTILE = 128


def n_tiles(V: int) -> int:
    return (V + VTILE - 1) // VTILE


def _logsumexp(a, axis=-1):
    """log sum exp along an axis, in binary64, shifted by the maximum."""
    a = np.asarray(a, dtype=np.float64)
    mx = np.max(a, axis=axis, keepdims=True)
    return np.squeeze(mx, axis=axis) + np.log(np.sum(np.exp(a - mx), axis=axis))


def head_logits(h, w):
    """logits[m, v] = sum_j h[m, j] w[v, j] in binary64; h [M, d], w [V, d]."""
    h = np.asarray(h, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    return h @ w.T


def head_logq(h, w):
    """Component log-probabilities log q(v | row m) in binary64, shape [M, V]."""
    logits = head_logits(h, w)
    return logits - _logsumexp(logits, axis=-1)[:, None]


def factor_logits(logits):
    """Split binary64 logits [M, V] into (tls, lmass, lse), all binary64."""
    logits = np.asarray(logits, dtype=np.float64)
    M, V = logits.shape
    nt = n_tiles(V)
    lmass = np.empty((M, nt), dtype=np.float64)
    tls = np.empty_like(logits)
    for t in range(nt):
        lo, hi = t * VTILE, min(V, (t + 1) * VTILE)
        lmass[:, t] = _logsumexp(logits[:, lo:hi], axis=-1)
        tls[:, lo:hi] = logits[:, lo:hi] - lmass[:, t:t + 1]
    lse = _logsumexp(logits, axis=-1)
    return tls, lmass, lse


def head_factored(h, w, v_chunk: int = 16384):
    """The head's output in the library's two-level form, rounded to binary32.

    Returns (tls [M, V], lmass [M, nT], lse [M]) as float32 arrays. Work is chunked over V
    (in multiples of the tile width) to bound memory; the arithmetic is unchanged.
    """
    h = np.asarray(h, dtype=np.float64)
    w = np.asarray(w)
    M = h.shape[0]
    V = w.shape[0]
    nt = n_tiles(V)
    v_chunk = max(VTILE, (v_chunk // VTILE) * VTILE)
    tls = np.empty((M, V), dtype=np.float32)
    lmass = np.empty((M, nt), dtype=np.float64)
    for lo in range(0, V, v_chunk):
        hi = min(V, lo + v_chunk)
        lg = h @ np.asarray(w[lo:hi], dtype=np.float64).T
        t_c, lm_c, _ = factor_logits(lg)
        tls[:, lo:hi] = t_c.astype(np.float32)
        lmass[:, lo // VTILE: lo // VTILE + lm_c.shape[1]] = lm_c
    lse = _logsumexp(lmass, axis=-1)
    return tls, lmass.astype(np.float32), lse.astype(np.float32)


def flat_logq(tls, lmass, lse):
    """fl32(tls + fl32(lmass - lse)) over the last axis; float32 out, same shape as tls."""
    tls = np.asarray(tls, dtype=np.float32)
    lmass = np.asarray(lmass, dtype=np.float32)
    lse = np.asarray(lse, dtype=np.float32)
    V = tls.shape[-1]
    off = (lmass - lse[..., None]).astype(np.float32)
    off_v = np.repeat(off, VTILE, axis=-1)[..., :V]
    return (tls + off_v).astype(np.float32)
