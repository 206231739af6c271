"""Pins of the oracle's greedy-branch proposal (appendix "Greedy-Branch Proposal",
"Prefix-Marginalized Conditional", "Distributional Correctness").

Each test checks the oracle against what the paper or the mathematics fixes: the joint
proposal written directly from its definition, closed forms for one category, the exact
emitted-token law, or a Monte Carlo law. None retypes the oracle's own formula.
"""

import numpy as np
from scipy import stats

from oracle import contract as C
from oracle import greedy as GR
from oracle import head as OH
from oracle import mixture as MX


def _logsoftmax(a):
    a = np.asarray(a, dtype=np.float64)
    m = a.max(-1, keepdims=True)
    return a - m - np.log(np.exp(a - m).sum(-1, keepdims=True))


def _branches_with_shared_prefixes(rng, K, R, V):
    """Branch tokens where several categories share initial tokens (a tree of branches)."""
    xhat = rng.integers(0, V, size=(K, R))
    for z in range(1, R):
        share = rng.integers(0, K)            # branch z copies the first `share` tokens of z - 1
        xhat[:share, z] = xhat[:share, z - 1]
    return xhat


def _joint(xhat_b, pi_b, x):
    """q_greedy(x_1..x_K) = sum_z pi_z prod_k 1{x_k = x_hat[k, z]} (Eq. greedy-branch-proposal)."""
    return sum(pi_b[z] for z in range(len(pi_b)) if np.array_equal(xhat_b[:, z], x))


def _prefix_joint(xhat_b, pi_b, x, n):
    """Marginal probability of the first n drafted tokens under the greedy proposal."""
    return sum(pi_b[z] for z in range(len(pi_b)) if np.array_equal(xhat_b[:n, z], x[:n]))


def test_branch_tokens_are_the_lowest_index_argmax_of_the_head():
    # One-hot hidden state e_j: logits are column j of w, chosen with a tie at the maximum.
    w = np.zeros((6, 3))
    w[:, 1] = [0.5, 2.0, -1.0, 2.0, 1.9, 0.0]
    h = np.array([[0.0, 1.0, 0.0]])
    assert GR.branch_tokens(OH.head_logits(h, w)).tolist() == [1]
    w[:, 1] = [3.0, 2.0, -1.0, 2.0, 1.9, 3.0]
    assert GR.branch_tokens(OH.head_logits(h, w)).tolist() == [0]


def test_block_draw_picks_the_drawn_branch_and_the_prior_law():
    rng = np.random.default_rng(5)
    K, R, V, N = 3, 4, 9, 20000
    xhat = np.broadcast_to(rng.integers(0, V, size=(K, R)), (N, K, R))
    ell = np.broadcast_to(rng.normal(size=R).astype(np.float32), (N, R))
    z, x = GR.sample_blocks_greedy(xhat, ell, 0.8, seed=11, step=2, seq=np.arange(N))
    assert np.array_equal(x, xhat[np.arange(N), :, z])
    pi = np.exp(ell[0].astype(np.float64) / np.float32(0.8))
    pi /= pi.sum()
    chi = stats.chisquare(np.bincount(z, minlength=R), pi * N)
    assert chi.pvalue > 1e-4


def test_conditional_chain_rule_equals_the_joint_by_enumeration():
    """prod_k q_greedy(x_k | x_<k) = q_greedy(x) for every branch block and for blocks that are
    no branch (zero), with branches sharing prefixes."""
    rng = np.random.default_rng(7)
    K, R, V = 4, 6, 5
    for trial in range(20):
        xhat = _branches_with_shared_prefixes(rng, K, R, V)
        ell = rng.normal(size=(1, R)).astype(np.float32)
        pi = MX.prior(ell, 1.0)[0]
        drafts = [xhat[:, z].copy() for z in range(R)]
        off = xhat[:, 0].copy()
        off[-1] = (off[-1] + 1) % V
        drafts.append(off)
        for x in drafts:
            out = GR.verify_blocks_greedy(xhat[None], ell, 1.0, x[None], np.zeros((1, K, V),
                                          np.float32), seed=1, step=0, seq=[0])
            prod = float(np.prod(out["q"][0]))
            want = _joint(xhat, pi, x)
            assert abs(prod - want) <= 1e-12 * max(want, 1e-300) + (0 if want else 1e-300)


def test_conditional_is_a_ratio_of_prefix_marginals_with_small_support():
    rng = np.random.default_rng(8)
    K, R, V = 5, 7, 4
    for trial in range(20):
        xhat = _branches_with_shared_prefixes(rng, K, R, V)
        ell = rng.normal(size=(1, R)).astype(np.float32)
        pi = MX.prior(ell, 0.6)[0]
        z0 = rng.integers(0, R)
        x = xhat[:, z0].copy()
        out = GR.verify_blocks_greedy(xhat[None], ell, 0.6, x[None],
                                      np.zeros((1, K, V), np.float32), seed=1, step=0, seq=[0])
        for k in range(K):
            want = _prefix_joint(xhat, pi, x, k + 1) / _prefix_joint(xhat, pi, x, k)
            assert abs(out["q"][0, k] - want) < 1e-13
            w = out["w"][0, k]
            support = {int(xhat[k, z]) for z in range(R) if w[z] > 0}
            consistent = [z for z in range(R) if np.array_equal(xhat[:k, z], x[:k])]
            assert len(support) <= len(consistent) <= R
            assert abs(w.sum() - 1.0) < 1e-14


def _r_interval_probs(w):
    """Exact probability of each index under inverse CDF with a uniform 32-bit word."""
    w = [int(v) for v in w]
    Z = sum(w)
    cum = np.cumsum([0] + w)
    edges = [-(-int(c) * 2**32 // Z) for c in cum]
    return np.diff(edges) / 2**32


def test_emitted_token_law_is_the_target_exactly():
    """Accepted mass plus residual gives exactly p at the first position, from the quantised
    integers the verifier uses (appendix "Distributional Correctness")."""
    rng = np.random.default_rng(9)
    R, V = 5, 8
    xhat = np.array([[1, 4, 1, 6, 4]])                     # K = 1, shared tokens 1 and 4
    ell = rng.normal(size=(1, R)).astype(np.float32)
    logp = _logsoftmax(rng.normal(size=(1, 1, V))).astype(np.float32)
    pi = MX.prior(ell, 1.0)[0]
    pz = _r_interval_probs(C.quant40(pi))                  # law of the drawn category
    draft = np.zeros(V)
    for z in range(R):
        draft[xhat[0, z]] += pz[z]
    qv = np.zeros(V)
    for z in range(R):
        qv[xhat[0, z]] += pi[z]
    q_int = C.quant40(qv)
    p_int = C.quant40(C.detexp32(logp[0, 0]))
    acc = np.array([min(2**32, -(-(int(p_int[v]) << 32) // int(q_int[v]))) / 2**32
                    if q_int[v] else 1.0 for v in range(V)])
    res = np.where(p_int > q_int, p_int - q_int, 0).astype(np.uint64)
    emitted = draft * acc + np.sum(draft * (1 - acc)) * _r_interval_probs(res)
    p = np.exp(logp[0, 0].astype(np.float64))
    np.testing.assert_allclose(emitted, p, atol=2e-6)
    # and the oracle's accept decisions realise that acceptance probability
    N = 4000
    out = GR.verify_blocks_greedy(np.broadcast_to(xhat[None], (N, 1, R)),
                                  np.broadcast_to(ell, (N, R)), 1.0,
                                  np.full((N, 1), 4), np.broadcast_to(logp, (N, 1, V)),
                                  seed=4, step=0, seq=np.arange(N))
    r = np.array([C.draw_u32(4, C.PURPOSE_ACCEPT, 0, s, 0) for s in range(N)])
    want = np.array([int(ri) * int(q_int[4]) < (int(p_int[4]) << 32) for ri in r])
    assert np.array_equal(out["n_accept"] == 1, want)


def test_single_category_closed_form():
    """R = 1: q_greedy is a point mass on the branch token, so beta_k = p_k(x_hat_k),
    A_k = p_k(x_hat_k) and E = AL = sum_i prod_{j<=i} p_j(x_hat_j)."""
    rng = np.random.default_rng(10)
    K, V = 6, 11
    xhat = rng.integers(0, V, size=(1, K, 1))
    logp = _logsoftmax(rng.normal(size=(1, K, V))).astype(np.float32)
    out = GR.verify_blocks_greedy(xhat, np.zeros((1, 1), np.float32), 1.0, xhat[:, :, 0], logp,
                                  seed=2, step=0, seq=[0])
    p = np.exp(logp[0, np.arange(K), xhat[0, :, 0]].astype(np.float64))
    np.testing.assert_allclose(out["q"][0], 1.0, rtol=0, atol=0)
    np.testing.assert_allclose(out["beta"][0], p, rtol=1e-15)
    want_E = sum(np.prod(p[:i + 1]) for i in range(K))
    assert abs(out["E"][0] - want_E) < 1e-14
    assert abs(out["al"][0] - want_E) < 1e-6 * want_E
    # along a trajectory that leaves the branch at position 2 the mass is zero afterwards
    xs = xhat[:, :, 0].copy()
    xs[0, 2] = (xs[0, 2] + 1) % V
    beta, E = GR.expected_len_greedy(xhat, np.zeros((1, 1), np.float32), 1.0, xs, logp)
    np.testing.assert_allclose(beta[0, :3], p[:3], rtol=1e-15)
    assert np.all(beta[0, 3:] == 0.0)


def test_zero_category_temperature_is_one_deterministic_block():
    rng = np.random.default_rng(12)
    K, R, V = 4, 5, 9
    xhat = rng.integers(0, V, size=(1, K, R))
    ell = np.array([[0.1, 2.0, 2.0, -1.0, 0.5]], np.float32)
    z, x = GR.sample_blocks_greedy(xhat, ell, 0.0, seed=3, step=0, seq=[0])
    assert z[0] == 1 and np.array_equal(x[0], xhat[0, :, 1])
    logp = _logsoftmax(rng.normal(size=(1, K, V))).astype(np.float32)
    out = GR.verify_blocks_greedy(xhat, ell, 0.0, x, logp, seed=3, step=0, seq=[0])
    assert np.all(out["q"][0] == 1.0)


def _exact_expected_accepted(xhat_b, pi_b, logp_b):
    """E[n_accept] = sum_z pi_z sum_i prod_{j<=i} min(1, p_j(x_j) / q(x_j | x_<j)) with
    x = branch z and the conditional taken as a ratio of prefix marginals."""
    K, R = xhat_b.shape
    total = 0.0
    for z in range(R):
        x = xhat_b[:, z]
        run, s = 1.0, 0.0
        for j in range(K):
            q = _prefix_joint(xhat_b, pi_b, x, j + 1) / _prefix_joint(xhat_b, pi_b, x, j)
            run *= min(1.0, float(np.exp(np.float64(logp_b[j, x[j]]))) / q)
            s += run
        total += pi_b[z] * s
    return total


def test_monte_carlo_accepted_length_and_first_token_law():
    rng = np.random.default_rng(13)
    K, R, V, N = 4, 4, 6, 1 << 14
    xhat1 = _branches_with_shared_prefixes(rng, K, R, V)
    ell1 = rng.normal(size=R).astype(np.float32)
    # target concentrated near the branches so that acceptance is substantial
    g = rng.normal(size=(K + 1, V))
    for z in range(R):
        g[np.arange(K), xhat1[:, z]] += 1.5
    logp1 = _logsoftmax(g).astype(np.float32)
    xhat = np.broadcast_to(xhat1, (N, K, R))
    ell = np.broadcast_to(ell1, (N, R))
    logp = np.broadcast_to(logp1, (N, K + 1, V))
    seq = np.arange(N)
    _, x = GR.sample_blocks_greedy(xhat, ell, 1.0, seed=21, step=5, seq=seq)
    out = GR.verify_blocks_greedy(xhat, ell, 1.0, x, logp, seed=21, step=5, seq=seq,
                                  with_beta=False)
    na = out["n_accept"].astype(np.float64)
    want = _exact_expected_accepted(xhat1, MX.prior(ell1[None], 1.0)[0], logp1)
    assert abs(na.mean() - want) < 5 * na.std() / np.sqrt(N)
    first = np.where(out["n_accept"] >= 1, x[:, 0], out["next_token"])
    p1 = np.exp(logp1[0].astype(np.float64))
    chi = stats.chisquare(np.bincount(first, minlength=V), p1 * N)
    assert chi.pvalue > 1e-4


def test_full_acceptance_draws_the_bonus_and_rejection_uses_the_residual():
    K, R, V = 3, 2, 5
    xhat = np.array([[[1, 1], [2, 3], [0, 4]]])
    ell = np.array([[0.0, 0.0]], np.float32)
    # target equal to the proposal at every position: everything is accepted
    logp = np.full((1, K + 1, V), -np.inf, np.float32)
    logp[0, 0, 1] = 0.0
    logp[0, 1, 2] = np.log(np.float32(0.5)); logp[0, 1, 3] = np.log(np.float32(0.5))
    logp[0, 2, 0] = 0.0
    logp[0, 3, 4] = 0.0
    out = GR.verify_blocks_greedy(xhat, ell, 1.0, np.array([[1, 2, 0]]), logp, seed=1, step=0,
                                  seq=[0])
    assert out["n_accept"][0] == 3 and out["next_token"][0] == 4
    # target puts no mass on the drafted token: rejected, residual is p itself
    logp2 = logp.copy()
    logp2[0, 0] = -np.inf
    logp2[0, 0, 3] = 0.0
    out = GR.verify_blocks_greedy(xhat, ell, 1.0, np.array([[1, 2, 0]]), logp2, seed=1, step=0,
                                  seq=[0])
    assert out["n_accept"][0] == 0 and out["next_token"][0] == 3


def test_bonus_token_follows_the_extra_target_row():
    """With the target equal to the (point-mass) proposal every position is accepted; the bonus
    is the contract's residual-purpose draw at counter K from the extra row, and follows it."""
    K, V, N = 3, 7, 6000
    rng = np.random.default_rng(14)
    xhat = np.broadcast_to(rng.integers(0, V, size=(1, K, 1)), (N, K, 1))
    logp = np.full((N, K + 1, V), -np.inf, np.float32)
    logp[:, np.arange(K), xhat[0, :, 0]] = 0.0
    bonus = _logsoftmax(rng.normal(size=V)).astype(np.float32)
    logp[:, K] = bonus
    seq = np.arange(N) + 50
    out = GR.verify_blocks_greedy(xhat, np.zeros((N, 1), np.float32), 1.0, xhat[:, :, 0], logp,
                                  seed=6, step=3, seq=seq, with_beta=False)
    assert np.all(out["n_accept"] == K)
    for b in range(0, N, 997):
        r = C.draw_u32(6, C.PURPOSE_RESIDUAL, K, int(seq[b]), 3)
        assert out["next_token"][b] == C.icdf(C.quant40(C.detexp32(bonus)), r)
    chi = stats.chisquare(np.bincount(out["next_token"], minlength=V),
                          np.exp(bonus.astype(np.float64)) * N)
    assert chi.pvalue > 1e-4
