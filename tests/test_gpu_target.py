"""GPU parity of dbl_target_logprobs and dbl_early_determinism against the oracle.

The kept set of every row (which ids are finite) must be identical: both cuts are integer
decisions on binary32 values computed the same way on both sides. Log-probabilities of kept ids
agree within 2e-6 (binary64 normaliser summed in a different order, stored as binary32).
"""
import time

import numpy as np
import pytest
import torch

import synth
from oracle import target as TG

pytestmark = pytest.mark.gpu


def _logits(N, V, seed, ties=False):
    if ties == "flat":   # every logit equal: top-k keeps the whole row
        return np.zeros((N, V), np.float32)
    g = synth.make_uniform_logits((N, V), seed, scale=3.0).numpy()
    perm = np.random.default_rng(seed).permutation(V)
    g = g - 1.1 * np.log1p(perm)[None, :]
    if ties == "ulp":   # the 40 largest logits one ulp apart: fl32(x / T) merges neighbours
        g = g.astype(np.float32)
        for r in range(N):
            top = np.argsort(-g[r])[:40]
            g[r, top] = np.float32(7.0) + np.arange(40, dtype=np.float32) * np.spacing(np.float32(7.0))
    elif ties == "tail":   # one token at 0, the rest ~27.5 below it, where the integer masses
        # are 0, 1 or 2: a nucleus with p near 1 cuts there, in a bin past 2000 (the kernel then
        # computes the masses in every pass, not the bins alone)
        g = (-27.5 + 0.15 * synth.make_uniform_logits((N, V), seed).numpy()).astype(np.float32)
        g[:, 0] = 0.0
    elif ties:   # coarse values: many equal logits at both cuts
        g = np.round(g * 2.0) / 2.0
    return g.astype(np.float32)


CASES = [
    # name, N, V, T, top_k, top_p, ties
    ("paper-t07-k20-p08", 6, 151936, 0.7, 20, 0.8, False),
    ("paper-t10-k20-p095", 6, 151936, 1.0, 20, 0.95, False),
    ("paper-t15-k20-p095", 6, 151936, 1.5, 20, 0.95, False),
    ("greedy", 5, 151936, 0.0, 20, 0.95, False),
    ("nucleus-only", 4, 151936, 1.0, 0, 0.9, False),
    ("top-k-only", 4, 50000, 1.0, 50, 1.0, False),
    ("no-filter", 3, 3001, 1.3, 0, 1.0, False),
    ("ties-at-both-cuts", 16, 2000, 1.0, 30, 0.7, True),
    ("ties-nucleus-only", 16, 2000, 1.0, 0, 0.5, True),
    ("tiny-vocab", 8, 7, 1.0, 3, 0.6, True),
    ("top-k-ragged-row", 4, 50001, 1.0, 50, 0.9, False),
    ("top-k-1000-ties", 4, 151936, 1.0, 1000, 0.9, True),
    ("top-k-1024", 3, 151936, 1.2, 1024, 0.95, False),
    ("top-k-1025", 3, 151936, 1.2, 1025, 0.95, False),
    ("flat-row-top-k", 2, 151936, 1.0, 20, 0.95, "flat"),
    ("one-ulp-neighbours-t15", 4, 30000, 1.5, 20, 0.95, "ulp"),
    ("one-ulp-neighbours-t07", 4, 30000, 0.7, 20, 0.95, "ulp"),
    ("temperature-3e4-merges-values", 4, 30000, 3e4, 20, 0.95, False),
    ("temperature-1e-3", 4, 30000, 1e-3, 20, 0.9, False),
    ("split-k256", 3, 151936, 1.0, 256, 0.95, False),
    ("split-k257", 3, 151936, 1.0, 257, 0.95, False),
    ("split-ties-overflow", 3, 151936, 1.0, 20, 0.95, True),
    ("split-smallest-vocab", 3, 16384, 1.0, 20, 0.95, False),
    ("split-ragged-vocab", 3, 16387, 1.0, 20, 0.95, False),
    ("nucleus-p0999", 3, 151936, 1.0, 0, 0.999, False),
    ("nucleus-p001", 3, 151936, 1.0, 0, 0.01, False),
    ("nucleus-high-T", 3, 151936, 5.0, 0, 0.9, False),
    ("nucleus-top-k-ge-V", 2, 3000, 1.0, 5000, 0.8, False),
    ("nucleus-ragged-vocab", 3, 50001, 0.7, 0, 0.8, False),
    ("flat-row-nucleus", 2, 151936, 1.0, 0, 0.95, "flat"),
    ("nucleus-cut-in-the-tail", 2, 151936, 1.0, 0, 0.9999999, "tail"),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_target_filter_parity(case):
    """Both launch forms (rows split over several workgroups through the workspace, and one
    workgroup per row) against the oracle, and bit-identical to each other."""
    from paper_2608_05448_amd import dblast as D
    name, N, V, T, k, p, ties = case
    print(f"[target] {name} N={N} V={V} T={T} k={k} p={p}", flush=True)
    lg = _logits(N, V, 7 + len(name), ties)
    lgd = torch.from_numpy(lg).cuda()
    got = D.dbl_target_logprobs(lgd, T, k, p)
    one = D.dbl_target_logprobs(lgd, T, k, p, split=False)
    torch.cuda.synchronize()
    assert torch.equal(got, one)
    got = got.cpu().numpy()
    want = TG.filter_logprobs(lg, T, k, p)
    assert np.array_equal(np.isfinite(got), np.isfinite(want))
    fin = np.isfinite(want)
    assert np.max(np.abs(got[fin] - want[fin])) < 2e-6
    print(f"[target] {name}: kept per row {np.isfinite(want).sum(1).tolist()}", flush=True)


def test_target_filter_benchmark_rows():
    """The Qwen3-8B verification rows (16 blocks x 17 positions) with the paper's filters."""
    from paper_2608_05448_amd import dblast as D
    N, V = 272, 151936
    lg = torch.from_numpy(_logits(N, V, 99)).cuda()
    out = torch.empty_like(lg)
    ws = torch.empty(D.dbl_workspace_bytes(D.DBL_OP_TARGET, N, 1, 1, 0, V), dtype=torch.uint8,
                     device="cuda")
    for T, k, p in ((0.7, 20, 0.8), (1.0, 20, 0.95), (1.5, 20, 1.0), (1.0, 0, 0.95)):
        for split in (True, False):
            D.dbl_target_logprobs(lg, T, k, p, out=out, ws=ws, split=split)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(5):
                D.dbl_target_logprobs(lg, T, k, p, out=out, ws=ws, split=split)
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t0) / 5 * 1e3
            print(f"[target] rows {N} x {V}, T={T} k={k} p={p} split={split}: {ms:.3f} ms "
                  f"({N * V * 8 / ms / 1e6:.0f} GB/s of logits in + logp out)", flush=True)
    rows = [0, 135, 271]
    want = TG.filter_logprobs(lg[rows].cpu().numpy(), 1.0, 0, 0.95)
    got = out[rows].cpu().numpy()
    assert np.array_equal(np.isfinite(got), np.isfinite(want))


def test_early_determinism_parity():
    from paper_2608_05448_amd import dblast as D
    M, b, V = 300, 8, 500
    lp = TG.filter_logprobs(_logits(M * b, V, 5), 1.0, 20, 0.9).reshape(M, b, V)
    rng = np.random.default_rng(6)
    p = np.exp(lp.astype(np.float64))
    cum = np.cumsum(p / p.sum(-1, keepdims=True), -1)
    x = np.minimum((cum < rng.random((M, b, 1))).sum(-1), V - 1).astype(np.int32)
    terms, mean = D.dbl_early_determinism(torch.from_numpy(x).cuda(), torch.from_numpy(lp).cuda())
    torch.cuda.synchronize()
    lpx = lp[np.arange(M)[:, None], np.arange(b)[None, :], x]
    want_terms = np.exp(np.cumsum(lpx.astype(np.float64), axis=1)).mean(1)
    np.testing.assert_allclose(terms.cpu().numpy(), want_terms, rtol=1e-6, atol=1e-9)
    assert abs(mean.item() - TG.early_determinism(lpx)) < 1e-6
