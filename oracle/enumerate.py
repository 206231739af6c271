"""Exact quantities by enumerating every block: CPU oracle for tiny V and K.

TEST INFRASTRUCTURE (see ``oracle/contract.py``).

These routines work directly from the joint proposal of Eq. cp-drafter,

    q(x_{1:i} | y) = sum_z q(z | y) prod_{j<=i} q_j(x_j | y, z),

(the marginal of the block joint on its first i positions), and take conditionals as ratios
of joints, Eq. proposal-conditional. They never form the category posterior, so they check
the posterior route of ``oracle/mixture.py`` rather than repeat it. The target is taken
prefix-independent, p_i(. | y, x_<i) = p_i(.), as in the synthetic workloads.

All arithmetic is binary64 on probabilities (q = exp(lq), p = exp(logp)), with no
quantisation. Sizes grow as V^K: keep V^K below a few million.
"""
from __future__ import annotations

import itertools

import numpy as np


def _prefix_tables(q, pi):
    """For i = 0..K, the joint J_i[x_1..x_i] = sum_z pi_z prod_{j<i} q_j(x_j|z) as a V^i array."""
    K, R, V = q.shape
    prods = np.ones((1, R))               # prod_{j<i} q_j(x_j | z) for every prefix, flattened
    tables = [np.array([1.0])]
    for i in range(K):
        prods = (prods[:, None, :] * q[i].T[None, :, :]).reshape(-1, R)
        tables.append(prods @ pi)
    return tables


def block_joint(q, pi):
    """q(x_{1:K}) for every block, shape [V] * K (Eq. cp-drafter)."""
    K, R, V = q.shape
    return _prefix_tables(q, pi)[K].reshape((V,) * K)


def conditional(q, pi, prefix, i):
    """q(. | x_<i) as a length-V vector by the ratio of joints, Eq. proposal-conditional."""
    K, R, V = q.shape
    prefix = list(prefix)[:i]
    num = np.zeros(V)
    den = 0.0
    for z in range(R):
        pz = pi[z] * np.prod([q[j, z, prefix[j]] for j in range(i)]) if i else pi[z]
        num += pz * q[i, z]
        den += pz
    return num / den if den > 0 else num


def exact_expected_al(q, pi, p):
    """E_{x ~ q}[AL_b(x)] by enumeration (left side of Eq. acceptance-length-objective).

    E[AL] = sum_l sum_{x_{1:l}} prod_{j<=l} min(p_j(x_j), q(x_j | x_<j)); the conditional is
    the ratio of consecutive prefix joints. q [K, R, V] probabilities, pi [R], p [K, V].
    """
    K, R, V = q.shape
    tables = _prefix_tables(q, pi)
    total = 0.0
    surv = np.array([1.0])                 # prod_{j<i} min(p_j, q(x_j | x_<j)) per prefix
    for i in range(K):
        num = tables[i + 1].reshape(-1, V)          # q(x_{1:i+1})
        den = tables[i][:, None]                    # q(x_{1:i})
        with np.errstate(divide="ignore", invalid="ignore"):
            cond = np.where(den > 0, num / np.where(den > 0, den, 1.0), 0.0)
        surv = (surv[:, None] * np.minimum(p[i][None, :], cond)).reshape(-1)
        total += surv.sum()
    return total


def expected_al_change_of_measure(q, pi, p):
    """Right side of Eq. acceptance-length-objective: sum_l E_{x ~ p}[r_l prod_{j<=l} A_j].

    r_l = q(x_{1:l}) / p(x_{1:l}) over target-sampled prefixes (p > 0) and
    A_j = min(1, p_j(x_j) / q(x_j | x_<j)).
    """
    K, R, V = q.shape
    tables = _prefix_tables(q, pi)
    total = 0.0
    pj = np.array([1.0])                   # p(x_{1:i}) per prefix
    accp = np.array([1.0])                 # prod_{j<i} A_j per prefix
    for i in range(K):
        num = tables[i + 1].reshape(-1, V)
        den = tables[i][:, None]
        with np.errstate(divide="ignore", invalid="ignore"):
            cond = np.where(den > 0, num / np.where(den > 0, den, 1.0), 0.0)
            a = np.where(cond > 0, np.minimum(1.0, p[i][None, :] / np.where(cond > 0, cond, 1.0)),
                         1.0)
        pj = (pj[:, None] * p[i][None, :]).reshape(-1)
        accp = (accp[:, None] * a).reshape(-1)
        qj = tables[i + 1]
        with np.errstate(divide="ignore", invalid="ignore"):
            r = np.where(pj > 0, qj / np.where(pj > 0, pj, 1.0), 0.0)
        total += np.sum(pj * r * accp)
    return total


def all_blocks(V, K):
    """Every block x_{1:K} in row-major order of the [V] * K joint array."""
    return np.array(list(itertools.product(range(V), repeat=K)), dtype=np.int64)
