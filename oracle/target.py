"""Target-side sampling transform and the early-determinism diagnostic: CPU oracle.

TEST INFRASTRUCTURE (see ``oracle/contract.py``): only tests, the smoke check and the benchmark's
CPU baseline use this module; the GPU library never does.

Target log-probabilities p(. | y, x_<i) are those of the target's sampling distribution: its
logits divided by the temperature, restricted by top-k and then top-p (nucleus) filtering and
renormalised (Sec. "Acceptance-Oriented Training": the same transform generates the training
trajectory and enters the acceptance probabilities; Sec. "Experiments": temperatures 0.7 to 1.5,
top-p 0.8 or 0.95, top-k 20). Outside the kept set the log-probability is -inf.

The paper does not spell out tie handling or the arithmetic of the nucleus cut; the reading used
here (and by the GPU library) is:

* temperature 0 keeps only the lowest-index maximum (log-probability 0 there);
* s(v) = fl32(logit(v) / T) in binary32;
* top-k (k > 0) keeps every v whose s(v) is at least the k-th largest value (ties at the cut are
  all kept);
* top-p (p < 1) on the kept set: with m the maximum and the integer masses
  P(v) = floor(detexp32(fl32(s(v) - m)) * 2^40) of the determinism contract, Z their sum over the
  kept set and T_p = ceil(p * Z) (binary64 product of the binary32 p), the kept tokens are visited by decreasing s
  and, among equal s, increasing id; a token is kept while the mass of the tokens before it is
  below T_p (the first token is always kept);
* log p(v) = s(v) - m - log(sum over kept u of exp(s(u) - m)) in binary64, stored as binary32.

The early-determinism diagnostic (appendix "Target-Block Early Determinism") of M sampled target
blocks of length b is  D_hat = 1/(M b) sum_m sum_j prod_{i<=j} p(x_i^(m) | y, x_<i^(m)),
an estimate of D_b = (1/b) sum_j sum_{u in V^j} p(u)^2 (the mean collision probability of the
target-prefix distributions).
"""
from __future__ import annotations

import numpy as np

from .contract import detexp32, quant40


def filter_logprobs(logits, temperature: float, top_k: int = 0, top_p: float = 1.0):
    """Filtered target log-probabilities, binary32 [N, V], for logits [N, V] (binary32)."""
    logits = np.asarray(logits, dtype=np.float32)
    N, V = logits.shape
    out = np.full((N, V), -np.inf, dtype=np.float32)
    if temperature == 0:
        out[np.arange(N), np.argmax(logits, axis=1)] = 0.0
        return out
    s = (logits / np.float32(temperature)).astype(np.float32)
    for n in range(N):
        row = s[n]
        keep = np.ones(V, dtype=bool)
        if top_k > 0 and top_k < V:
            kth = np.sort(row)[::-1][top_k - 1]
            keep = row >= kth
        m = row[keep].max()
        if top_p < 1.0:
            idx = np.nonzero(keep)[0]
            order = idx[np.lexsort((idx, -row[idx].astype(np.float64)))]
            P = quant40(detexp32((row[order] - m).astype(np.float32))).astype(object)
            Z = int(sum(P))
            Tp = max(1, int(np.ceil(np.float64(np.float32(top_p)) * np.float64(Z))))
            before = 0
            kept = []
            for v, pv in zip(order, P):
                if before >= Tp:
                    break
                kept.append(v)
                before += int(pv)
            keep = np.zeros(V, dtype=bool)
            keep[np.array(kept)] = True
        sel = row[keep].astype(np.float64) - np.float64(m)
        lse = np.log(np.sum(np.exp(sel)))
        out[n, keep] = (sel - lse).astype(np.float32)
    return out


def early_determinism(logp_x):
    """D_hat from the gathered target log-probabilities of M sampled blocks: logp_x [M, b] with
    logp_x[m, i] = log p(x_i^(m) | y, x_<i^(m)). Returns the scalar estimate (binary64)."""
    lp = np.asarray(logp_x, dtype=np.float64)
    M, b = lp.shape
    return float(np.sum(np.exp(np.cumsum(lp, axis=1))) / (M * b))
