"""Pins of the training-objective oracle (Eqs. block-nll, independent-nll, dependent-nll,
acceptance-length-objective, subblock-objective).

The prefix likelihoods and conditionals are checked against exact enumeration of the block joint
(``oracle/enumerate.py`` builds it from Eq. cp-drafter without the log-domain mixture), the
change-of-measure identity is checked term by term, and the truncation and surrogate against
hand-computed cases.
"""
import itertools
import math

import numpy as np

from oracle import enumerate as EN
from oracle import mixture as MX
from oracle import objective as OB


def _logsoftmax(a):
    a = np.asarray(a, dtype=np.float64)
    m = a.max(-1, keepdims=True)
    return a - m - np.log(np.exp(a - m).sum(-1, keepdims=True))


def _case(seed, K, R, V):
    rng = np.random.default_rng(seed)
    lq = _logsoftmax(rng.normal(size=(K, R, V)) * 1.3).astype(np.float32)
    ell = rng.normal(size=(1, R)).astype(np.float32)
    logp = _logsoftmax(rng.normal(size=(K, V))).astype(np.float32)
    return lq, ell, logp


def _all_blocks(V, K):
    return np.array(list(itertools.product(range(V), repeat=K)), dtype=np.int64)


def test_nll_and_prefix_likelihoods_match_enumeration():
    K, R, V = 3, 4, 5
    lq, ell, logp = _case(1, K, R, V)
    q = np.exp(lq.astype(np.float64))
    pi = MX.prior(ell, 1.0)[0]
    X = _all_blocks(V, K)
    n = len(X)
    out = OB.acceptance_objective(np.broadcast_to(lq, (n, K, R, V)), np.broadcast_to(ell, (n, R)),
                                  1.0, X, np.broadcast_to(logp, (n, K, V)))
    joint = EN.block_joint(q, pi)
    prefix = EN._prefix_tables(q, pi)          # marginals of the first l tokens, V^l each
    for i, x in enumerate(X):
        assert abs(out["nll"][i] + math.log(joint[tuple(x)])) < 1e-12
        for l in range(1, K + 1):
            marg = prefix[l].reshape((V,) * l)[tuple(x[:l])]
            assert abs(out["log_q"][i, l - 1] - math.log(marg)) < 1e-12
            cond = EN.conditional(q, pi, x, l - 1)[x[l - 1]]
            want_A = min(1.0, math.exp(float(logp[l - 1, x[l - 1]])) / cond)
            assert abs(out["A"][i, l - 1] - want_A) < 1e-12


def test_single_category_nll_is_the_sum_of_cross_entropies():
    """R = 1 gives Eq. independent-nll: -sum_i log q_i(x*_i)."""
    K, V = 6, 9
    rng = np.random.default_rng(2)
    lq = _logsoftmax(rng.normal(size=(1, K, 1, V))).astype(np.float32)
    xs = rng.integers(0, V, size=(1, K))
    out = OB.acceptance_objective(lq, np.zeros((1, 1), np.float32), 1.0, xs,
                                  np.zeros((1, K, V), np.float32))
    want = -sum(float(lq[0, j, 0, xs[0, j]]) for j in range(K))
    assert abs(out["nll"][0] - want) < 1e-12


def test_change_of_measure_term_by_term():
    """For every prefix length l: E_{x~q}[prod_{j<=l} A_j] = E_{x~p}[r_l prod_{j<=l} A_j]
    (Eq. acceptance-length-objective), and their sum over l is the exact E[AL]."""
    K, R, V = 3, 3, 4
    lq, ell, logp = _case(3, K, R, V)
    q = np.exp(lq.astype(np.float64))
    pi = MX.prior(ell, 1.0)[0]
    p = np.exp(logp.astype(np.float64))
    prefix = EN._prefix_tables(q, pi)
    total = 0.0
    for l in range(1, K + 1):
        P = _all_blocks(V, l)                    # every prefix of length l, padded with 0
        X = np.concatenate([P, np.zeros((len(P), K - l), np.int64)], axis=1)
        n = len(X)
        out = OB.acceptance_objective(np.broadcast_to(lq, (n, K, R, V)),
                                      np.broadcast_to(ell, (n, R)), 1.0, X,
                                      np.broadcast_to(logp, (n, K, V)))
        qj = prefix[l]                           # q(x_{1:l}) in the same (row-major) order
        pj = np.prod(p[np.arange(l)[None, :], P], axis=1)
        prodA = np.prod(out["A"][:, :l], axis=1)
        lhs = np.sum(qj * prodA)
        rhs = np.sum(pj * np.exp(out["log_r"][:, l - 1]) * prodA)
        assert abs(lhs - rhs) < 1e-12
        total += lhs
    assert abs(total - EN.exact_expected_al(q, pi, p)) < 1e-12


def test_identical_proposal_and_target_give_log_factorial():
    """q = p (R = 1): every A_j = 1 and r_l = 1, so S_l = l, l_tau = K and J = log K!."""
    K, V = 5, 7
    rng = np.random.default_rng(4)
    lp = _logsoftmax(rng.normal(size=(1, K, V))).astype(np.float32)
    xs = rng.integers(0, V, size=(1, K))
    out = OB.acceptance_objective(lp[:, :, None, :], np.zeros((1, 1), np.float32), 1.0, xs, lp)
    np.testing.assert_allclose(out["S"][0], np.arange(1, K + 1), atol=1e-12)
    assert out["ell_tau"][0] == K
    assert abs(out["J"][0] - math.log(math.factorial(K))) < 1e-12


def test_truncation_stops_at_the_first_small_ratio():
    """R = 1, q = p except q_3(x*_3) = p_3(x*_3) / 20: r = (1, 1, 0.05, 0.05) so l_tau = 3,
    A = (1, 1, 1, 1), S = (1, 2, 3, 4) and J = log 1 + log 2 + (log 0.05 + log 3)."""
    K, V = 4, 3
    lp = np.log(np.full((1, K, V), 1.0 / V)).astype(np.float32)
    xs = np.array([[0, 1, 2, 0]])
    lq = np.array(lp)[:, :, None, :].copy()
    q3 = np.array([1.0 / 60, 0.0, 0.0])
    q3[1:] = (1 - q3[0]) / 2
    lq[0, 2, 0] = np.log(np.roll(q3, 2)).astype(np.float32)   # q_3(x*_3 = 2) = 1/60
    out = OB.acceptance_objective(lq, np.zeros((1, 1), np.float32), 1.0, xs, lp)
    r = np.exp(out["log_r"][0])
    np.testing.assert_allclose(r, [1, 1, 0.05, 0.05], rtol=1e-6)
    assert out["ell_tau"][0] == 3
    np.testing.assert_allclose(out["S"][0], [1, 2, 3, 4], rtol=1e-6)
    assert abs(out["J"][0] - (math.log(2) + math.log(0.05) + math.log(3))) < 1e-6
    # tau below every ratio keeps the whole block; tau above every ratio keeps one term
    assert OB.acceptance_objective(lq, np.zeros((1, 1), np.float32), 1.0, xs, lp,
                                   tau=0.01)["ell_tau"][0] == K
    assert OB.acceptance_objective(lq, np.zeros((1, 1), np.float32), 1.0, xs, lp,
                                   tau=10.0)["ell_tau"][0] == 1


def test_accepted_prefix_sums_multiply_acceptance_probabilities():
    """R = 1, q = p except q_2(x*_2) = 2 p_2(x*_2): A = (1, 1/2, 1, 1), so
    S = (1, 1 + 1/2, 1 + 1/2 + 1/2, 1 + 3/2) and r = (1, 2, 2, 2)."""
    K, V = 4, 4
    lp = np.log(np.full((1, K, V), 1.0 / V)).astype(np.float32)
    xs = np.array([[3, 0, 1, 2]])
    lq = np.array(lp)[:, :, None, :].copy()
    q2 = np.full(V, (1 - 0.5) / (V - 1))
    q2[0] = 0.5                                                # q_2(x*_2 = 0) = 2 p_2
    lq[0, 1, 0] = np.log(q2).astype(np.float32)
    out = OB.acceptance_objective(lq, np.zeros((1, 1), np.float32), 1.0, xs, lp)
    np.testing.assert_allclose(out["A"][0], [1, 0.5, 1, 1], rtol=1e-6)
    np.testing.assert_allclose(out["S"][0], [1, 1.5, 2.0, 2.5], rtol=1e-6)
    np.testing.assert_allclose(np.exp(out["log_r"][0]), [1, 2, 2, 2], rtol=1e-6)
    assert out["ell_tau"][0] == K
