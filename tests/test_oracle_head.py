"""Pins of the oracle's output head (logits through the shared LM head, log-softmax over V)."""
import numpy as np
import pytest

from oracle import head as H


def test_onehot_hidden_states_give_closed_form_probabilities():
    """With h[m] = e_{j(m)} and w[:, j] = log c_v, q(v | m) = c_v / sum_u c_u exactly."""
    rng = np.random.default_rng(0)
    M, d, V = 5, 7, 300
    cols = [3, 0, 6, 3, 1]                      # which hidden unit each row selects
    counts = rng.integers(1, 50, size=(d, V))   # positive integers c[j, v]
    w = np.log(counts.T.astype(np.float64))     # [V, d]
    h = np.zeros((M, d))
    for m, j in enumerate(cols):
        h[m, j] = 1.0
    logq = H.head_logq(h, w)
    for m, j in enumerate(cols):
        want = np.log(counts[j] / counts[j].sum())
        np.testing.assert_allclose(logq[m], want, rtol=0, atol=1e-12)


def test_logq_is_normalised_and_non_positive():
    rng = np.random.default_rng(1)
    h = rng.normal(size=(9, 33))
    w = rng.normal(size=(517, 33)) * 0.5
    logq = H.head_logq(h, w)
    assert np.all(logq <= 1e-15)
    np.testing.assert_allclose(np.exp(logq).sum(-1), 1.0, rtol=0, atol=1e-12)


@pytest.mark.parametrize("V", [1, 127, 128, 129, 300, 1000])
def test_factored_form_identities(V):
    """Per-tile probabilities sum to 1, tile masses sum to 1, and tls + lmass - lse = log q."""
    rng = np.random.default_rng(V)
    h = rng.normal(size=(4, 16))
    w = rng.normal(size=(V, 16))
    logits = H.head_logits(h, w)
    tls, lmass, lse = H.factor_logits(logits)
    nt = H.n_tiles(V)
    assert lmass.shape == (4, nt)
    for t in range(nt):
        lo, hi = t * 128, min(V, (t + 1) * 128)
        np.testing.assert_allclose(np.exp(tls[:, lo:hi]).sum(-1), 1.0, atol=1e-12)
    np.testing.assert_allclose(np.exp(lmass - lse[:, None]).sum(-1), 1.0, atol=1e-12)
    rebuilt = tls + np.repeat(lmass, 128, axis=1)[:, :V] - lse[:, None]
    np.testing.assert_allclose(rebuilt, H.head_logq(h, w), atol=1e-12)


def test_binary32_flat_logq_within_rounding_bound():
    """fl32(tls + fl32(lmass - lse)) is within a few binary32 ulps of the binary64 log q."""
    rng = np.random.default_rng(5)
    d, V = 64, 1000
    h = rng.normal(size=(6, d)).astype(np.float32)
    w = (rng.normal(size=(V, d)) / np.sqrt(d)).astype(np.float32)
    tls, lmass, lse = H.head_factored(h, w, v_chunk=256)
    flat = H.flat_logq(tls, lmass, lse).astype(np.float64)
    exact = H.head_logq(h, w)
    # Three binary32 roundings (tls, lmass - lse, the sum) of magnitudes below 16.
    bound = 3 * 16 * 2.0**-24
    assert np.max(np.abs(flat - exact)) < bound
    # The chunked and unchunked factorisations agree.
    t2, l2, s2 = H.head_factored(h, w, v_chunk=100000)
    np.testing.assert_array_equal(tls, t2)
    np.testing.assert_array_equal(lmass, l2)


def test_rows_and_vocabulary_are_not_transposed():
    """Row m of the output depends on row m of h only and column v on row v of w only."""
    rng = np.random.default_rng(9)
    h = rng.normal(size=(3, 8))
    w = rng.normal(size=(11, 8))
    base = H.head_logits(h, w)
    h2 = h.copy()
    h2[1] += 1.0
    changed = np.any(H.head_logits(h2, w) != base, axis=1)
    assert changed.tolist() == [False, True, False]
    w2 = w.copy()
    w2[7] *= 2.0
    changed = np.any(H.head_logits(h, w2) != base, axis=0)
    assert changed.tolist() == [v == 7 for v in range(11)]
