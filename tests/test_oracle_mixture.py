"""Pins of the oracle's prior, block draw, posterior, verifier and expected length.

Each test checks the oracle against something the paper or the mathematics fixes (a closed
form, an identity, an exact enumeration, a textbook special case or a law checked by a
chi-square test), never against a retyped copy of its own formula.
"""
import math

import numpy as np
import pytest
from scipy import stats

from oracle import contract as C
from oracle import enumerate as EN
from oracle import mixture as MX


def _logsoftmax(a):
    a = np.asarray(a, dtype=np.float64)
    m = a.max(-1, keepdims=True)
    return a - m - np.log(np.exp(a - m).sum(-1, keepdims=True))


def tiny_case(seed, B, K, R, V, q_scale=1.0, p_scale=2.0, kp_extra=1):
    rng = np.random.default_rng(seed)
    lq = _logsoftmax(rng.normal(size=(K, R, V)) * q_scale).astype(np.float32)
    lq = np.broadcast_to(lq, (B, K, R, V))
    ell = np.broadcast_to(rng.normal(size=R).astype(np.float32), (B, R))
    logp = _logsoftmax(rng.normal(size=(K + kp_extra, V)) * p_scale).astype(np.float32)
    logp = np.broadcast_to(logp, (B, K + kp_extra, V))
    return lq, ell, logp


def _probs(lq):
    return np.exp(np.asarray(lq, dtype=np.float64))


def _one_tile(lq):
    """The two-level form of rows that fit one 128-id tile: tls = lq, lmass = lse = 0."""
    lq = np.asarray(lq, dtype=np.float32)
    assert lq.shape[-1] <= MX.TILE
    return lq, np.zeros(lq.shape[:-1] + (1,), np.float32), np.zeros(lq.shape[:-1], np.float32)


# ---------------------------------------------------------------------------------------
# Prior
# ---------------------------------------------------------------------------------------
def test_prior_closed_form():
    zt = 0.7
    ell = (zt * np.log([[1.0, 2.0, 3.0, 4.0]])).astype(np.float32)
    pi = MX.prior(ell, zt)
    np.testing.assert_allclose(pi[0], [0.1, 0.2, 0.3, 0.4], rtol=0, atol=2e-7)
    assert abs(pi.sum() - 1.0) < 1e-15


def test_prior_zero_temperature_single_category_and_scaling():
    ell = np.array([[0.3, 1.5, 1.5, -2.0]], dtype=np.float32)
    assert MX.prior(ell, 0.0)[0].tolist() == [0.0, 1.0, 0.0, 0.0]   # lowest-index argmax
    assert MX.prior(np.array([[4.2]], np.float32), 0.9)[0].tolist() == [1.0]
    rng = np.random.default_rng(2)
    ell = rng.normal(size=(5, 6)).astype(np.float32)
    for zt in (0.25, 1.0, 3.0):
        want = np.exp(ell.astype(np.float64) / np.float32(zt))
        want /= want.sum(-1, keepdims=True)
        np.testing.assert_allclose(MX.prior(ell, zt), want, rtol=1e-14)
    with pytest.raises(ValueError):
        MX.prior(ell, -0.1)


# ---------------------------------------------------------------------------------------
# Posterior and the prefix-marginalised conditional
# ---------------------------------------------------------------------------------------
def test_posterior_matches_product_form_and_sums_to_one():
    """w_{k,z} = q(z) prod_{j<k} q_j(x_j|z) / sum_z' (...), Eq. category-posterior."""
    B, K, R, V = 6, 5, 4, 9
    lq, ell, logp = tiny_case(11, B, K, R, V)
    rng = np.random.default_rng(12)
    x = rng.integers(0, V, size=(B, K))
    out = MX.verify_blocks(lq, ell, 0.8, x, logp, seed=0, step=0, seq=np.arange(B))
    pi = np.exp(ell[0].astype(np.float64) / np.float32(0.8))
    pi /= pi.sum()
    q = _probs(lq[0])
    for b in range(B):
        for k in range(K):
            num = pi * np.prod([q[j, :, x[b, j]] for j in range(k)], axis=0) if k else pi.copy()
            np.testing.assert_allclose(out["w"][b, k], num / num.sum(), rtol=1e-12)
            assert abs(out["w"][b, k].sum() - 1.0) < 1e-14


def test_chain_rule_by_enumeration():
    """prod_k q(x_k | x_<k) via the posterior equals the block joint of Eq. cp-drafter."""
    K, R, V = 3, 3, 4
    blocks = EN.all_blocks(V, K)
    B = blocks.shape[0]
    lq, ell, logp = tiny_case(21, B, K, R, V)
    out = MX.verify_blocks(lq, ell, 1.3, blocks, logp, seed=0, step=0, seq=np.arange(B),
                           with_beta=False)
    q = _probs(lq[0])
    chain = np.ones(B)
    for k in range(K):
        qx = q[k][:, blocks[:, k]].T                      # [B, R]
        chain *= np.sum(out["w"][:, k] * qx, axis=1)
    pi = MX.prior(ell[:1], 1.3)[0]
    joint = EN.block_joint(q, pi).reshape(-1)
    np.testing.assert_allclose(chain, joint, rtol=1e-12)
    # The conditional used by verification is the ratio-of-joints conditional.
    for b in (0, 17, B - 1):
        for k in range(K):
            mix = np.sum(out["w"][b, k][:, None] * q[k], axis=0)
            np.testing.assert_allclose(mix, EN.conditional(q, pi, blocks[b], k), rtol=1e-12)


def test_acceptance_mass_is_one_minus_total_variation():
    """beta_1 = sum_v min(p, q) = (sum p + sum q - sum |p - q|) / 2 = 1 - TV(p, q)."""
    B, K, R, V = 3, 2, 3, 50
    lq, ell, logp = tiny_case(31, B, K, R, V)
    x = np.zeros((B, K), dtype=np.int64)
    out = MX.verify_blocks(lq, ell, 1.0, x, logp, seed=0, step=0, seq=np.arange(B))
    pi = MX.prior(ell[:1], 1.0)[0]
    q0 = np.sum(pi[:, None] * _probs(lq[0, 0]), axis=0)
    p0 = _probs(logp[0, 0])
    identity = 0.5 * (p0.sum() + q0.sum() - np.abs(p0 - q0).sum())
    np.testing.assert_allclose(out["beta"][:, 0], identity, rtol=1e-13)
    np.testing.assert_allclose(out["beta"][:, 0], 1.0 - 0.5 * np.abs(p0 - q0).sum(), atol=1e-6)


# ---------------------------------------------------------------------------------------
# Block draw
# ---------------------------------------------------------------------------------------
def _chi2_pvalue(counts, probs):
    counts = np.asarray(counts, dtype=np.float64)
    probs = np.asarray(probs, dtype=np.float64)
    keep = probs > 0
    assert counts[~keep].sum() == 0
    exp = probs[keep] / probs[keep].sum() * counts.sum()
    return stats.chisquare(counts[keep], exp).pvalue


def test_block_draw_law_is_the_mixture_joint():
    """Two-stage draw (z, then positions in parallel) samples Eq. cp-drafter."""
    K, R, V, N = 2, 2, 3, 8000
    lq, ell, _ = tiny_case(41, N, K, R, V, q_scale=1.5)
    z, x = MX.sample_blocks(*_one_tile(lq), ell, 1.0, seed=5, step=2, seq=np.arange(N))
    pi = MX.prior(ell[:1], 1.0)[0]
    assert _chi2_pvalue(np.bincount(z, minlength=R), pi) > 1e-4
    joint = EN.block_joint(_probs(lq[0]), pi).reshape(-1)
    cells = np.bincount(x[:, 0] * V + x[:, 1], minlength=V * V)
    assert _chi2_pvalue(cells, joint) > 1e-4


def test_single_category_reduces_to_independent_block_sampling():
    K, V, N = 2, 4, 8000
    lq, ell, _ = tiny_case(43, N, K, 1, V, q_scale=1.5)
    z, x = MX.sample_blocks(*_one_tile(lq), ell, 1.0, seed=9, step=0, seq=np.arange(N))
    assert np.all(z == 0)
    q = _probs(lq[0, :, 0])
    cells = np.bincount(x[:, 0] * V + x[:, 1], minlength=V * V)
    assert _chi2_pvalue(cells, np.outer(q[0], q[1]).reshape(-1)) > 1e-4


def _two_level(logits):
    """Binary32 two-level form of binary64 logits [..., V] (tile log-prob, tile log-mass,
    log-sum-exp), built here from the definitions of a tile-wise log-softmax."""
    lg = np.asarray(logits, dtype=np.float64)
    V = lg.shape[-1]
    nT = -(-V // MX.TILE)
    lmass = np.stack([np.log(np.exp(lg[..., t * MX.TILE:(t + 1) * MX.TILE]).sum(-1))
                      for t in range(nT)], -1)
    tls = lg - np.repeat(lmass, MX.TILE, axis=-1)[..., :V]
    lse = np.log(np.exp(lg).sum(-1))
    return tls.astype(np.float32), lmass.astype(np.float32), lse.astype(np.float32)


def _token_law(tls_row, lmass_row, lse):
    """Exact law of MX.draw_token over both 32-bit words: the tile's interval probability
    times the id's within the tile."""
    off = (np.asarray(lmass_row, np.float32) - np.float32(lse)).astype(np.float32)
    pt = _r_interval_probs(C.quant40(C.detexp32(off)))
    law = np.zeros(len(tls_row))
    for t, ptt in enumerate(pt):
        ids = np.asarray(tls_row[t * MX.TILE:(t + 1) * MX.TILE], np.float32)
        law[t * MX.TILE:t * MX.TILE + len(ids)] = ptt * _r_interval_probs(
            C.quant40(C.detexp32(ids)))
    return law


@pytest.mark.parametrize("V", [128, 300, 1000])
def test_two_stage_token_law_is_the_softmax(V):
    """Drawing the tile from its mass, then the id within it, has the law softmax(logits) of
    the whole row: within the binary32 rounding of the two-level form (relative), and within
    the 2^-32 resolution of an inverse CDF driven by one 32-bit word, per stage (absolute)."""
    rng = np.random.default_rng(V)
    logits = rng.normal(size=V) * 3.0
    logits[rng.integers(0, V, 5)] += 6.0   # a few dominant ids, in different tiles
    q = np.exp(logits - logits.max())
    q /= q.sum()
    law = _token_law(*_two_level(logits))
    assert abs(law.sum() - 1.0) < 1e-12
    np.testing.assert_allclose(law, q, rtol=2e-6, atol=2 * 2.0 ** -32)


def test_two_stage_draw_uses_both_words_and_the_tile_offset():
    """Monte Carlo over many sequences: multi-tile rows give chi-square-consistent tokens, and
    the ids drawn inside a tile follow its within-tile law (word 1 independent of word 0)."""
    K, R, V, N = 1, 2, 300, 30000
    rng = np.random.default_rng(7)
    logits = rng.normal(size=(K, R, V)) * 1.5
    tls, lmass, lse = _two_level(logits)
    B = N
    b3 = lambda a: np.broadcast_to(a, (B,) + a.shape)
    ell = np.broadcast_to(np.array([0.3, -0.2], np.float32), (B, R))
    z, x = MX.sample_blocks(b3(tls), b3(lmass), b3(lse), ell, 1.0, seed=19, step=5,
                            seq=np.arange(N) + 7)
    pi = MX.prior(ell[:1], 1.0)[0]
    assert _chi2_pvalue(np.bincount(z, minlength=R), pi) > 1e-4
    for zz in range(R):
        sel = z == zz
        q = np.exp(logits[0, zz] - logits[0, zz].max())
        assert _chi2_pvalue(np.bincount(x[sel, 0], minlength=V), q / q.sum()) > 1e-4


def test_two_stage_draw_single_tile_is_the_flat_inverse_cdf():
    """A row of one tile: the tile stage is certain, so the token is the flat inverse CDF of
    its quantised masses with word 1."""
    rng = np.random.default_rng(3)
    lq = _logsoftmax(rng.normal(size=100)).astype(np.float32)
    for s in range(50):
        r1 = C.draw_u32_word1(4, C.PURPOSE_TOKEN, 0, s, 2)
        got = MX.draw_token(lq, np.zeros(1, np.float32), np.float32(0), C.draw_u32(
            4, C.PURPOSE_TOKEN, 0, s, 2), r1)
        assert got == C.icdf(C.quant40(C.detexp32(lq)), r1)


# ---------------------------------------------------------------------------------------
# Verification laws
# ---------------------------------------------------------------------------------------
def _r_interval_probs(weights):
    """Exact probability of each index under icdf with a uniform 32-bit r."""
    w = [int(v) for v in weights]
    Z = sum(w)
    cum = np.cumsum([0] + w)
    edges = [-(-int(c) * 2**32 // Z) for c in cum]
    return np.diff(edges) / 2**32


def test_emitted_token_law_is_the_target_exactly():
    """Accepted mass min(p, q) plus the residual supplies exactly p (Sec. Distributional
    correctness), computed from the quantised integer quantities the verifier uses."""
    R, V = 3, 7
    lq, ell, logp = tiny_case(51, 1, 1, R, V, q_scale=1.2, p_scale=1.0, kp_extra=0)
    pi = MX.prior(ell, 1.0)[0]
    pz = _r_interval_probs(C.quant40(pi))                          # law of the category
    y = C.detexp32(lq[0, 0])                                        # [R, V]
    draft = sum(pz[z] * _r_interval_probs(C.quant40(y[z])) for z in range(R))
    Q = np.zeros(V)
    for z in range(R):
        Q = Q + pi[z] * y[z].astype(np.float64)
    q_int = C.quant40(Q)
    p_int = C.quant40(C.detexp32(logp[0, 0]))
    acc = np.array([min(2**32, -(-(int(p_int[v]) << 32) // int(q_int[v]))) / 2**32
                    if q_int[v] else 1.0 for v in range(V)])
    res = np.where(p_int > q_int, p_int - q_int, 0).astype(np.uint64)
    emitted = draft * acc + np.sum(draft * (1 - acc)) * _r_interval_probs(res)
    p = _probs(logp[0, 0])
    np.testing.assert_allclose(emitted, p, atol=2e-6)
    assert np.abs(emitted - p).sum() < 5e-6


def test_emitted_tokens_follow_the_target_monte_carlo():
    """First emitted token ~ p_1 and, after an accepted first token, the second ~ p_2."""
    K, R, V, N = 2, 3, 5, 12000
    lq, ell, logp = tiny_case(53, N, K, R, V, q_scale=1.0, p_scale=1.0)
    seq = np.arange(N)
    _, x = MX.sample_blocks(*_one_tile(lq), ell, 1.0, seed=3, step=1, seq=seq)
    out = MX.verify_blocks(lq, ell, 1.0, x, logp, seed=3, step=1, seq=seq, with_beta=False)
    na, nt = out["n_accept"], out["next_token"]
    first = np.where(na >= 1, x[:, 0], nt)
    assert _chi2_pvalue(np.bincount(first, minlength=V), _probs(logp[0, 0])) > 1e-4
    sel = na >= 1
    second = np.where(na[sel] >= 2, x[sel, 1], nt[sel])
    assert sel.sum() > 2000
    assert _chi2_pvalue(np.bincount(second, minlength=V), _probs(logp[0, 1])) > 1e-4


def _textbook_speculative_sampling(lq1, logp, x, seed, step, seq):
    """Standard speculative sampling (Leviathan et al.; Chen et al.) with an independent
    proposal q_k, under the same random-number and quantisation contract."""
    K, V = lq1.shape
    n = 0
    for k in range(K):
        q_int = C.quant40(C.detexp32(lq1[k]))
        p_int = C.quant40(C.detexp32(logp[k]))
        r = C.draw_u32(seed, C.PURPOSE_ACCEPT, k, seq, step)
        if C.accept_int(r, q_int[x[k]], p_int[x[k]]):
            n += 1
            continue
        res = np.where(p_int > q_int, p_int - q_int, 0).astype(np.uint64)
        r = C.draw_u32(seed, C.PURPOSE_RESIDUAL, k, seq, step)
        t = C.icdf(res, r)
        return n, (t if t >= 0 else C.icdf(p_int, r))
    if logp.shape[0] > K:
        r = C.draw_u32(seed, C.PURPOSE_RESIDUAL, K, seq, step)
        return n, C.icdf(C.quant40(C.detexp32(logp[K])), r)
    return n, -1


def test_single_category_verify_is_textbook_speculative_sampling():
    K, V, N = 4, 6, 400
    rng = np.random.default_rng(61)
    lq = _logsoftmax(rng.normal(size=(N, K, 1, V)) * 0.7).astype(np.float32)
    logp = _logsoftmax(rng.normal(size=(N, K + 1, V)) * 0.7).astype(np.float32)
    ell = rng.normal(size=(N, 1)).astype(np.float32)
    seq = np.arange(N) + 1000
    _, x = MX.sample_blocks(*_one_tile(lq), ell, 1.0, seed=77, step=4, seq=seq)
    out = MX.verify_blocks(lq, ell, 1.0, x, logp, seed=77, step=4, seq=seq, with_beta=False)
    for b in range(N):
        n, t = _textbook_speculative_sampling(lq[b, :, 0], logp[b], x[b], 77, 4, int(seq[b]))
        assert (int(out["n_accept"][b]), int(out["next_token"][b])) == (n, t)
    assert 0 < out["n_accept"].mean() < K


def test_zero_target_probability_rejects():
    B, K, R, V = 4, 3, 2, 8
    lq, ell, logp = tiny_case(71, B, K, R, V)
    logp = np.array(logp)
    x = np.tile(np.array([[2, 5, 1]]), (B, 1))
    logp[:, 1, 5] = -np.inf
    out = MX.verify_blocks(lq, ell, 1.0, x, logp, seed=1, step=0, seq=np.arange(B))
    assert np.all(out["A"][:, 1] == 0.0)
    assert np.all(out["n_accept"] <= 1)
    # A correction drawn at position 1 comes from max(p - q, 0), which is 0 where p is.
    assert np.all(out["next_token"][out["n_accept"] == 1] != 5)


def test_full_acceptance_draws_the_bonus_token():
    """p = q accepts every position (u < 1 always); the bonus comes from the extra row."""
    B, K, V = 5, 4, 10
    rng = np.random.default_rng(81)
    lq = _logsoftmax(rng.normal(size=(B, K, 1, V))).astype(np.float32)
    logp = np.concatenate([lq[:, :, 0], _logsoftmax(rng.normal(size=(B, 1, V))).astype(np.float32)], 1)
    ell = np.zeros((B, 1), np.float32)
    seq = np.arange(B)
    _, x = MX.sample_blocks(*_one_tile(lq), ell, 1.0, seed=2, step=0, seq=seq)
    out = MX.verify_blocks(lq, ell, 1.0, x, logp, seed=2, step=0, seq=seq)
    assert np.all(out["n_accept"] == K)
    np.testing.assert_allclose(out["al"], K)
    for b in range(B):
        r = C.draw_u32(2, C.PURPOSE_RESIDUAL, K, b, 0)
        assert out["next_token"][b] == C.icdf(C.quant40(C.detexp32(logp[b, K])), r)
    out2 = MX.verify_blocks(lq, ell, 1.0, x, logp[:, :K], seed=2, step=0, seq=seq)
    assert np.all(out2["next_token"] == -1)


def test_zero_category_temperature_keeps_one_branch():
    B, K, R, V = 3, 4, 5, 12
    lq, ell, logp = tiny_case(91, B, K, R, V)
    top = int(np.argmax(ell[0]))
    z, x = MX.sample_blocks(*_one_tile(lq), ell, 0.0, seed=4, step=0, seq=np.arange(B))
    assert np.all(z == top)
    out = MX.verify_blocks(lq, ell, 0.0, x, logp, seed=4, step=0, seq=np.arange(B))
    want = np.zeros(R)
    want[top] = 1.0
    for k in range(K):
        np.testing.assert_array_equal(out["w"][:, k], np.tile(want, (B, 1)))


# ---------------------------------------------------------------------------------------
# Expected accepted length
# ---------------------------------------------------------------------------------------
def test_single_category_expected_length_closed_form():
    """R = 1 and a prefix-independent target: E[AL] = sum_i prod_{j<=i} (1 - TV(p_j, q_j))."""
    K, V = 4, 6
    lq, ell, logp = tiny_case(101, 1, K, 1, V, kp_extra=0)
    q = _probs(lq[0, :, 0])
    p = _probs(logp[0])
    beta_cf = 0.5 * (p.sum(1) + q.sum(1) - np.abs(p - q).sum(1))
    closed = np.sum(np.cumprod(beta_cf))
    exact = EN.exact_expected_al(_probs(lq[0]), np.array([1.0]), p)
    np.testing.assert_allclose(exact, closed, rtol=1e-12)
    xs = np.array([[1, 4, 0, 2]])
    beta, E = MX.expected_len_blocks(lq, ell, 1.0, xs, logp)
    np.testing.assert_allclose(E[0], closed, rtol=1e-12)


def test_change_of_measure_identity_by_enumeration():
    """Eq. acceptance-length-objective: the q-side and p-side sums agree exactly."""
    K, R, V = 3, 3, 6
    lq, ell, logp = tiny_case(111, 1, K, R, V, kp_extra=0)
    pi = MX.prior(ell, 1.0)[0]
    q, p = _probs(lq[0]), _probs(logp[0])
    a = EN.exact_expected_al(q, pi, p)
    b = EN.expected_al_change_of_measure(q, pi, p)
    np.testing.assert_allclose(a, b, rtol=1e-12)
    assert 0.1 < a < K


def test_expected_len_equals_verify_acceptance_mass_along_the_draft():
    B, K, R, V = 4, 5, 3, 20
    lq, ell, logp = tiny_case(121, B, K, R, V, kp_extra=0)
    rng = np.random.default_rng(122)
    x = rng.integers(0, V, size=(B, K))
    out = MX.verify_blocks(lq, ell, 0.6, x, logp, seed=0, step=0, seq=np.arange(B))
    beta, E = MX.expected_len_blocks(lq, ell, 0.6, x, logp)
    np.testing.assert_array_equal(beta, out["beta"])
    np.testing.assert_array_equal(E, out["E"])


def test_monte_carlo_accepted_length_matches_enumeration():
    """Brute-force E[AL] over all V^K blocks equals the mean accepted length of the sampler
    followed by the verifier (z-test at 5 standard errors)."""
    K, R, V, N = 4, 3, 8, 16384
    lq, ell, logp = tiny_case(131, N, K, R, V, q_scale=1.2, p_scale=1.2, kp_extra=0)
    pi = MX.prior(ell[:1], 1.0)[0]
    exact = EN.exact_expected_al(_probs(lq[0]), pi, _probs(logp[0]))
    seq = np.arange(N)
    _, x = MX.sample_blocks(*_one_tile(lq), ell, 1.0, seed=11, step=3, seq=seq)
    out = MX.verify_blocks(lq, ell, 1.0, x, logp, seed=11, step=3, seq=seq, with_beta=False)
    for sample in (out["n_accept"].astype(np.float64), out["al"]):
        se = sample.std(ddof=1) / math.sqrt(N)
        assert abs(sample.mean() - exact) < 5 * se, (sample.mean(), exact, se)
    assert exact > 0.3
