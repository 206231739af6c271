"""GPU parity of the greedy-branch mode: the head's per-row argmax, dbl_sample_greedy,
dbl_verify_greedy and dbl_expected_len_greedy against the oracle.

The draw and the verifier receive the same branch tokens, category logits and target
log-probabilities on both sides: category, drafted tokens, accepted count and residual/bonus
token must match bit for bit; acceptance masses, AL_b and E within 1e-4 relative. The head's
argmax is compared with the oracle's binary64 argmax; a disagreement is allowed only where the two
candidates' binary64 logits lie within the fp32 accumulation error (certified near-tie).
"""
import zlib

import numpy as np
import pytest
import torch

import synth
from cases import np32
from oracle import greedy as GR
from oracle import head as OH

pytestmark = pytest.mark.gpu


def _rel_close(got, want, rtol=1e-4, floor=1e-30):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    mask = np.abs(want) > floor
    if mask.any():
        rel = np.max(np.abs(got[mask] - want[mask]) / np.abs(want[mask]))
        assert rel < rtol, rel
    assert np.all(np.abs(got[~mask]) < 1e-20)


def _check_argmax(got, logits64, tol):
    want = GR.branch_tokens(logits64)
    rows = np.nonzero(got != want)[0]
    for m in rows:
        gap = abs(logits64[m, got[m]] - logits64[m, want[m]])
        assert gap <= tol, (m, got[m], want[m], gap)
    return len(rows)


HEAD_CASES = [
    # name, B, K, R, d, V, dtype
    ("f32-tiny", 1, 4, 2, 64, 256, torch.float32),
    ("f32-ragged", 2, 3, 5, 40, 1001, torch.float32),
    ("bf16-dma", 2, 4, 8, 256, 3000, torch.bfloat16),
    ("bf16-register-staged", 1, 5, 7, 72, 777, torch.bfloat16),
    ("bf16-many-tiles", 4, 16, 8, 128, 20000, torch.bfloat16),
]


@pytest.mark.parametrize("case", HEAD_CASES, ids=[c[0] for c in HEAD_CASES])
def test_head_argmax_matches_oracle_and_leaves_logprobs_unchanged(case):
    from paper_2608_05448_amd import dblast as D
    name, B, K, R, d, V, dt = case
    print(f"[greedy head] {name} B={B} K={K} R={R} d={d} V={V}", flush=True)
    seed = zlib.crc32(name.encode()) % 1000
    h = synth.make_uniform_logits((B, K, R, d), seed + 1).to(dt)
    w = (synth.make_uniform_logits((V, d), seed + 2) * (3.0 / d ** 0.5)).to(dt)
    # exact ties at the maximum of row 0: a duplicated best row in the same tile and in another
    w64 = np32(w).astype(np.float64)
    h0 = np32(h).reshape(-1, d)[0].astype(np.float64)
    best = int(np.argmax(w64 @ h0))
    for dup in sorted({(best + 3) % V, (best + 300) % V} - {best}):
        w[dup] = w[best]
    hd, wd = h.cuda(), w.cuda()
    t1, l1, s1 = D.dbl_head_logprobs(hd, wd)
    t2, l2, s2, am = D.dbl_head_logprobs(hd, wd, argmax=True)
    torch.cuda.synchronize()
    assert torch.equal(t1, t2) and torch.equal(l1, l2) and torch.equal(s1, s2)
    logits = OH.head_logits(np32(h).reshape(-1, d), np32(w))
    got = am.cpu().numpy().reshape(-1)
    tol = 2e-5 if dt == torch.float32 else 2e-4
    _check_argmax(got, logits, tol)
    dups = [v for v in range(V) if np.array_equal(np32(w)[v], np32(w)[best])]
    if len(dups) > 1 and logits[0, best] == logits[0].max():
        assert got[0] == min(dups)


def _greedy_inputs(B, K, R, V, seed, share=True, aligned=True, kp_extra=1):
    rng = np.random.default_rng(seed)
    xhat = rng.integers(0, V, size=(B, K, R)).astype(np.int32)
    if share:   # branches that share initial tokens
        for z in range(1, R):
            n = rng.integers(0, K + 1, size=B)
            for b in range(B):
                xhat[b, :n[b], z] = xhat[b, :n[b], z - 1]
    ell = rng.normal(size=(B, R)).astype(np.float32)
    g = rng.normal(size=(B, K + kp_extra, V)) * 2.0
    if aligned:  # target mass on the branch tokens so that acceptance is exercised
        for z in range(R):
            g[np.arange(B)[:, None], np.arange(K)[None, :], xhat[:, :, z]] += 3.0 + z % 3
    logp = (g - np.log(np.exp(g - g.max(-1, keepdims=True)).sum(-1, keepdims=True))
            - g.max(-1, keepdims=True)).astype(np.float32)
    return xhat, ell, logp


GREEDY_CASES = [
    # name, B, K, R, V, z_temp, seed, step, seq_offset, kp_extra, share, aligned
    ("shared-prefixes-bonus", 8, 6, 4, 3000, 1.0, 0, 0, 0, 1, True, True),
    ("independent-target", 8, 6, 4, 3000, 0.7, 1, 2, 11, 0, False, False),
    ("zero-cat-temp", 6, 5, 5, 1000, 0.0, 2, 1, 0, 1, True, True),
    ("single-category", 10, 7, 1, 500, 1.0, 3, 0, 5, 1, False, True),
    ("full-vocab", 3, 16, 8, 151936, 1.0, 2**33 + 1, 4, 1000, 1, True, True),
    ("tiny-vocab", 5, 4, 3, 7, 1.3, 4, 0, 0, 1, True, True),
    ("ragged-vocab", 4, 5, 6, 1001, 1.0, 5, 3, 7, 1, True, True),
    ("max-categories", 3, 4, 64, 700, 1.0, 6, 0, 0, 1, True, True),
    ("many-blocks", 96, 8, 4, 2000, 1.0, 7, 9, 4321, 1, True, True),
    # The chain stages its gathers in LDS only for K <= 64 and K * R <= 1024; these two take the
    # unstaged walk (K * R > 1024, and K > 64).
    ("unstaged-wide", 4, 20, 64, 800, 1.0, 8, 0, 0, 1, True, True),
    ("unstaged-long", 3, 80, 4, 600, 1.0, 9, 2, 0, 1, True, True),
]


@pytest.mark.parametrize("case", GREEDY_CASES, ids=[c[0] for c in GREEDY_CASES])
def test_greedy_sample_verify_parity(case):
    from paper_2608_05448_amd import dblast as D
    name, B, K, R, V, zt, seed, step, so, kx, share, aligned = case
    print(f"[greedy] {name} B={B} K={K} R={R} V={V} seed={seed}", flush=True)
    xhat, ell, logp = _greedy_inputs(B, K, R, V, zlib.crc32(name.encode()) % 1000, share,
                                     aligned, kx)
    xd = torch.from_numpy(xhat).cuda()
    ed = torch.from_numpy(ell).cuda()
    ld = torch.from_numpy(logp).cuda()
    seq = so + np.arange(B)
    z_g, x_g = D.dbl_sample_greedy(xd, ed, z_temp=zt, seed=seed, step=step, seq_offset=so, V=V)
    torch.cuda.synchronize()
    z_o, x_o = GR.sample_blocks_greedy(xhat, ell, zt, seed, step, seq)
    np.testing.assert_array_equal(z_g.cpu().numpy(), z_o)
    np.testing.assert_array_equal(x_g.cpu().numpy(), x_o)
    out = D.dbl_verify_greedy(xd, ed, x_g, ld, z_temp=zt, seed=seed, step=step, seq_offset=so)
    torch.cuda.synchronize()
    ref = GR.verify_blocks_greedy(xhat, ell, zt, x_o, logp, seed, step, seq)
    np.testing.assert_array_equal(out["n_accept"].cpu().numpy(), ref["n_accept"])
    np.testing.assert_array_equal(out["next_token"].cpu().numpy(), ref["next_token"])
    _rel_close(out["accept_mass"].cpu().numpy(), ref["beta"])
    _rel_close(out["al_expected"].cpu().numpy(), ref["al"])
    _rel_close(out["exp_len"].cpu().numpy(), ref["E"])
    # a draft that leaves every branch (perturbed tokens) exercises empty consistent sets
    xbad = x_o.copy()
    xbad[:, K // 2] = (xbad[:, K // 2] + 1) % V
    out = D.dbl_verify_greedy(xd, ed, torch.from_numpy(xbad).cuda(), ld, z_temp=zt, seed=seed,
                              step=step, seq_offset=so)
    ref = GR.verify_blocks_greedy(xhat, ell, zt, xbad, logp, seed, step, seq)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out["n_accept"].cpu().numpy(), ref["n_accept"])
    np.testing.assert_array_equal(out["next_token"].cpu().numpy(), ref["next_token"])
    _rel_close(out["accept_mass"].cpu().numpy(), ref["beta"])
    # expected length along the (first K rows of the) target as a trajectory
    xs = np.argmax(logp[:, :K], axis=-1).astype(np.int32)
    beta_g, e_g = D.dbl_expected_len_greedy(xd, ed, torch.from_numpy(xs).cuda(),
                                            torch.from_numpy(np.ascontiguousarray(logp[:, :K])).cuda(),
                                            z_temp=zt)
    torch.cuda.synchronize()
    beta_o, e_o = GR.expected_len_greedy(xhat, ell, zt, xs, logp[:, :K])
    _rel_close(beta_g.cpu().numpy(), beta_o)
    _rel_close(e_g.cpu().numpy(), e_o)


def test_greedy_accept_paths_are_exercised():
    from paper_2608_05448_amd import dblast as D
    B, K, R, V = 256, 6, 4, 500
    xhat, ell, logp = _greedy_inputs(B, K, R, V, 99)
    xd, ed, ld = (torch.from_numpy(a).cuda() for a in (xhat, ell, logp))
    _, x = D.dbl_sample_greedy(xd, ed, seed=3, V=V)
    out = D.dbl_verify_greedy(xd, ed, x, ld, seed=3)
    na = out["n_accept"].cpu().numpy()
    assert (na == 0).any() and ((na > 0) & (na < K)).any() and (na == K).any()


def test_greedy_end_to_end_from_the_head_argmax():
    """Head argmax -> greedy draw -> verification; the oracle consumes the GPU's branch tokens."""
    from paper_2608_05448_amd import dblast as D
    B, K, R, d, V = 4, 8, 4, 128, 5000
    h = synth.make_uniform_logits((B, K, R, d), 31).to(torch.bfloat16)
    w = (synth.make_uniform_logits((V, d), 32) * (4.0 / d ** 0.5)).to(torch.bfloat16)
    ell = synth.make_uniform_logits((B, R), 33).to(torch.float32)
    _, _, _, am = D.dbl_head_logprobs(h.cuda(), w.cuda(), argmax=True)
    xhat = am.cpu().numpy()
    rng = np.random.default_rng(34)
    g = rng.normal(size=(B, K + 1, V)) * 2.0
    g[np.arange(B)[:, None], np.arange(K)[None, :], xhat[:, :, 0]] += 6.0
    logp = (g - np.log(np.exp(g).sum(-1, keepdims=True))).astype(np.float32)
    z, x = D.dbl_sample_greedy(am, ell.cuda(), seed=8, step=2, V=V)
    out = D.dbl_verify_greedy(am, ell.cuda(), x, torch.from_numpy(logp).cuda(), seed=8, step=2)
    torch.cuda.synchronize()
    z_o, x_o = GR.sample_blocks_greedy(xhat, ell.numpy(), 1.0, 8, 2, np.arange(B))
    ref = GR.verify_blocks_greedy(xhat, ell.numpy(), 1.0, x_o, logp, 8, 2, np.arange(B))
    np.testing.assert_array_equal(z.cpu().numpy(), z_o)
    np.testing.assert_array_equal(x.cpu().numpy(), x_o)
    np.testing.assert_array_equal(out["n_accept"].cpu().numpy(), ref["n_accept"])
    np.testing.assert_array_equal(out["next_token"].cpu().numpy(), ref["next_token"])


def test_greedy_random_shapes_against_the_oracle():
    """A seeded sweep of small random greedy-branch shapes (staged and unstaged chains, V below
    one tile, shared or independent branch prefixes, with and without the bonus row) against
    the oracle."""
    from paper_2608_05448_amd import dblast as D
    rng = np.random.default_rng(20261203)
    for i in range(14):
        B = int(rng.integers(1, 24))
        K = int(rng.integers(1, 40))
        R = int(rng.integers(1, 40))
        V = int(rng.choice([int(rng.integers(2, 128)), int(rng.integers(128, 5000))]))
        kx = int(rng.integers(0, 2))
        share, aligned = bool(rng.integers(0, 2)), bool(rng.integers(0, 2))
        zt = float(rng.choice([0.0, 0.5, 1.0, 2.0]))
        seed, step, so = int(rng.integers(0, 2**40)), int(rng.integers(0, 1000)), int(rng.integers(0, 999))
        print(f"[greedy random] {i}: B={B} K={K} R={R} V={V} Kp=K+{kx} share={share} "
              f"aligned={aligned} z_temp={zt} seed={seed} step={step} so={so}", flush=True)
        xhat, ell, logp = _greedy_inputs(B, K, R, V, 200 + i, share, aligned, kx)
        xd, ed, ld = (torch.from_numpy(a).cuda() for a in (xhat, ell, logp))
        seq = so + np.arange(B)
        z_g, x_g = D.dbl_sample_greedy(xd, ed, z_temp=zt, seed=seed, step=step, seq_offset=so, V=V)
        out = D.dbl_verify_greedy(xd, ed, x_g, ld, z_temp=zt, seed=seed, step=step, seq_offset=so)
        torch.cuda.synchronize()
        z_o, x_o = GR.sample_blocks_greedy(xhat, ell, zt, seed, step, seq)
        np.testing.assert_array_equal(z_g.cpu().numpy(), z_o)
        np.testing.assert_array_equal(x_g.cpu().numpy(), x_o)
        ref = GR.verify_blocks_greedy(xhat, ell, zt, x_o, logp, seed, step, seq)
        np.testing.assert_array_equal(out["n_accept"].cpu().numpy(), ref["n_accept"])
        np.testing.assert_array_equal(out["next_token"].cpu().numpy(), ref["next_token"])
        _rel_close(out["accept_mass"].cpu().numpy(), ref["beta"])
        _rel_close(out["al_expected"].cpu().numpy(), ref["al"])
        _rel_close(out["exp_len"].cpu().numpy(), ref["E"])
