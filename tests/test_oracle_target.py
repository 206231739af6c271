"""Pins of the target-transform and early-determinism oracle."""
import math

import numpy as np

from oracle import target as TG


def test_no_filter_is_the_tempered_softmax():
    rng = np.random.default_rng(1)
    logits = (rng.normal(size=(4, 50)) * 3).astype(np.float32)
    for T in (0.7, 1.0, 1.5):
        got = TG.filter_logprobs(logits, T).astype(np.float64)
        s = (logits / np.float32(T)).astype(np.float64)
        want = s - s.max(1, keepdims=True)
        want -= np.log(np.exp(want).sum(1, keepdims=True))
        np.testing.assert_allclose(got, want, atol=2e-6)
        np.testing.assert_allclose(np.exp(got.astype(np.float64)).sum(1), 1.0, atol=1e-5)


def test_zero_temperature_is_one_hot_at_the_lowest_maximum():
    logits = np.array([[0.5, 2.0, 2.0, -1.0]], np.float32)
    assert TG.filter_logprobs(logits, 0.0)[0].tolist() == [-np.inf, 0.0, -np.inf, -np.inf]


def test_top_k_keeps_the_k_largest_and_ties_at_the_cut():
    rng = np.random.default_rng(2)
    logits = rng.permutation(np.arange(40, dtype=np.float32))[None, :]
    got = TG.filter_logprobs(logits, 1.0, top_k=7)
    kept = np.nonzero(np.isfinite(got[0]))[0]
    assert sorted(logits[0, kept].tolist()) == list(range(33, 40))
    # renormalised over the kept set
    want = logits[0, kept].astype(np.float64)
    want = want - np.log(np.exp(want).sum())
    np.testing.assert_allclose(got[0, kept], want, atol=2e-6)
    tied = np.array([[5.0, 3.0, 4.0, 3.0, 1.0, 3.0]], np.float32)
    kept = np.isfinite(TG.filter_logprobs(tied, 1.0, top_k=3)[0])
    assert kept.tolist() == [True, True, True, True, False, True]   # 5, 4 and every 3


def test_top_p_keeps_the_smallest_prefix_reaching_p():
    # probabilities proportional to 8, 4, 2, 1, 1 (sum 16), listed out of order
    probs = np.array([2, 8, 1, 4, 1], dtype=np.float64) / 16
    logits = np.log(probs).astype(np.float32)[None, :]
    def kept(p, k=0):
        return np.nonzero(np.isfinite(TG.filter_logprobs(logits, 1.0, top_k=k, top_p=p)[0]))[0].tolist()
    assert kept(0.3) == [1]                 # 8/16 already reaches 0.3
    assert kept(0.7) == [1, 3]              # 8/16 < 0.7 <= 12/16
    assert kept(0.8) == [0, 1, 3]           # 12/16 < 0.8 <= 14/16
    assert kept(0.99) == [0, 1, 2, 3, 4]
    assert kept(0.99, k=2) == [1, 3]        # top-k first, then top-p on the renormalised rest
    got = TG.filter_logprobs(logits, 1.0, top_p=0.8)[0]
    np.testing.assert_allclose(np.exp(got[[1, 3, 0]].astype(np.float64)), [8 / 14, 4 / 14, 2 / 14],
                               atol=1e-6)
    # equal probabilities at the cut are taken in increasing id order
    flat = np.zeros((1, 6), np.float32)
    assert np.nonzero(np.isfinite(TG.filter_logprobs(flat, 1.0, top_p=0.4)[0]))[0].tolist() == [0, 1, 2]


def test_early_determinism_closed_form_and_monte_carlo():
    """With a prefix-independent target, E[prod_{i<=j} p_i(x_i)] = prod_{i<=j} sum_v p_i(v)^2,
    so D_b = (1/b) sum_j prod_{i<=j} sum_v p_i(v)^2; a one-hot target gives 1."""
    b, V, M = 4, 6, 200000
    assert TG.early_determinism(np.zeros((10, b))) == 1.0
    rng = np.random.default_rng(3)
    p = rng.dirichlet(np.ones(V) * 0.5, size=b)
    want = np.mean(np.cumprod((p ** 2).sum(1)))
    x = np.stack([rng.choice(V, size=M, p=p[i]) for i in range(b)], axis=1)
    lp = np.log(p[np.arange(b)[None, :], x])
    terms = np.exp(np.cumsum(lp, axis=1)).mean(1)
    got = TG.early_determinism(lp)
    assert abs(got - want) < 5 * terms.std() / math.sqrt(M)
