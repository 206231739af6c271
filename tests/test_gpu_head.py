"""GPU parity of dbl_head_logprobs against the oracle head (binary64 GEMM + log-softmax).

Tolerances: 2e-5 absolute on log-probabilities for fp32 inputs and 2e-3 for bf16 inputs with
fp32 accumulation (both sides read the identical bf16 values).
"""
import math

import numpy as np
import pytest
import torch

import synth
from cases import flat_from_factored, np32
from oracle import head as OH

pytestmark = pytest.mark.gpu


def _run(h, w):
    from paper_2608_05448_amd import dblast as D
    out = D.dbl_head_logprobs(h.cuda(), w.cuda())
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in out]


def _check(h, w, tol, label):
    B, K, R, d = h.shape
    V = w.shape[0]
    print(f"[head] {label} B={B} K={K} R={R} d={d} V={V} dtype={h.dtype}", flush=True)
    tls, lmass, lse = _run(h, w)
    hh, ww = np32(h).reshape(-1, d), np32(w)
    ref = OH.head_logq(hh, ww)
    got = flat_from_factored(tls.reshape(-1, V), lmass.reshape(-1, lmass.shape[-1]),
                             lse.reshape(-1)).astype(np.float64)
    err = np.max(np.abs(got - ref))
    print(f"[head] {label} max |log q error| = {err:.3e}", flush=True)
    assert err < tol
    # The factored parts individually.
    r_tls, r_lm, r_lse = OH.factor_logits(OH.head_logits(hh, ww))
    assert np.max(np.abs(tls.reshape(-1, V) - r_tls)) < tol
    assert np.max(np.abs(lmass.reshape(-1, lmass.shape[-1]) - r_lm)) < tol
    assert np.max(np.abs(lse.reshape(-1) - r_lse)) < tol


def test_head_fp32_tiny_workload():
    wl = synth.WORKLOADS["tiny"]
    _check(synth.make_h(wl), synth.make_w(wl), 2e-5, "tiny")


@pytest.mark.parametrize("B,K,R,d,V", [
    (3, 2, 5, 100, 1000),    # d not a multiple of 8 (fp32 path allows it), ragged last tile
    (1, 1, 1, 1, 1),         # smallest problem
    (2, 3, 7, 40, 129),      # one id in the last tile
])
def test_head_fp32_ragged(B, K, R, d, V):
    h = synth.make_uniform_logits((B, K, R, d), 11).to(torch.float32)
    w = (synth.make_uniform_logits((V, d), 12) / math.sqrt(d)).to(torch.float32)
    _check(h, w, 2e-5, "fp32-ragged")


@pytest.mark.parametrize("B,K,R,d,V", [
    (3, 2, 5, 136, 1000),    # hidden size not a multiple of the 32-wide K step; ragged tiles
    (2, 10, 15, 512, 5000),  # several branch-row and vocabulary tiles, ragged on both
    (1, 4, 5, 64, 1001),     # V % 4 != 0: scalar stores
    (1, 1, 5, 8, 77),        # fewer ids than one tile
    (4, 16, 8, 256, 2048),   # exact tile multiples
    (2, 3, 5, 96, 3001),     # hidden size a multiple of 32 but not 64: direct-to-LDS kernel
    (1, 16, 8, 192, 4100),   # three 64-deep stages (odd count) in the register-staged kernel
    (9, 16, 8, 128, 3000),   # five branch-row tiles: more than one group of the tile order
    (9, 16, 8, 96, 3000),    # the same with the direct-to-LDS kernel
    (1, 1, 3, 64, 270000),   # more than 2048 tiles per row: the LSE pass reads the row twice
    (65, 16, 16, 64, 600),   # 65 branch-row tiles: the tile order's groups of 8, a partial last group
])
def test_head_bf16_ragged(B, K, R, d, V):
    h = synth.make_uniform_logits((B, K, R, d), 21).to(torch.bfloat16)
    w = (synth.make_uniform_logits((V, d), 22) * 0.05).to(torch.bfloat16)
    _check(h, w, 2e-3, "bf16-ragged")


def test_head_bf16_qwen3_8b_all_rows():
    """Full Qwen3-8B-shaped head (the benchmark's launch), every row against the oracle."""
    _full_size("qwen3_8b")


def test_head_bf16_qwen3_4b_all_rows():
    """Full Qwen3-4B-shaped head in the benchmark's launch, every row against the oracle."""
    _full_size("qwen3_4b")


def _full_size(name):
    from cases import oracle_full_head
    from paper_2608_05448_amd import dblast as D
    wl = synth.WORKLOADS[name]
    print(f"[head] full-size {name} M={wl.M} d={wl.d} V={wl.V}", flush=True)
    h = synth.make_h(wl, "cuda")
    w = synth.make_w(wl, "cuda")
    tls, lmass, lse = D.dbl_head_logprobs(h, w)
    torch.cuda.synchronize()
    M, V, nT = wl.M, wl.V, OH.n_tiles(wl.V)
    t2 = tls.view(M, V)
    # Identities at every row: each tile's probabilities sum to 1, tile masses sum to 1.
    tile_sums = torch.exp(t2.view(M, nT, 128).double()).sum(-1)   # V = 1187 * 128 exactly
    assert torch.max(torch.abs(tile_sums - 1.0)).item() < 1e-5
    mass = torch.exp((lmass.view(M, nT) - lse.view(M, 1)).double()).sum(-1)
    assert torch.max(torch.abs(mass - 1.0)).item() < 1e-5
    assert torch.max(t2).item() <= 1e-6
    del tile_sums, mass
    print(f"[head] full-size {name}: oracle head on all {M} rows", flush=True)
    ref = oracle_full_head(name, h, w)
    lm2, ls2 = lmass.view(M, nT), lse.view(M)
    err = 0.0
    for r0 in range(0, M, 256):
        got = flat_from_factored(t2[r0:r0 + 256].cpu().numpy(), lm2[r0:r0 + 256].cpu().numpy(),
                                 ls2[r0:r0 + 256].cpu().numpy())
        err = max(err, float(np.max(np.abs(got.astype(np.float64) - ref[r0:r0 + 256]))))
    print(f"[head] full-size {name} all rows max |log q error| = {err:.3e}", flush=True)
    assert err < 2e-3


def test_head_random_shapes():
    """A seeded sweep of random head shapes in both input precisions: hidden sizes that take each
    bf16 kernel (d % 64 = 0, d % 32 = 0 only, d % 8 = 0 only) and arbitrary fp32 ones, branch-row
    and vocabulary counts with ragged last tiles."""
    rng = np.random.default_rng(20261204)
    for i in range(12):
        bf16 = i % 3 != 2
        B, K, R = int(rng.integers(1, 25)), int(rng.integers(1, 9)), int(rng.integers(1, 9))
        if bf16:
            d = int(rng.choice([64 * int(rng.integers(1, 9)), 32 * int(rng.integers(1, 17)),
                                8 * int(rng.integers(1, 65))]))
        else:
            d = int(rng.integers(1, 300))
        V = int(rng.choice([int(rng.integers(1, 130)), int(rng.integers(130, 6000))]))
        dt = torch.bfloat16 if bf16 else torch.float32
        h = synth.make_uniform_logits((B, K, R, d), 300 + i).to(dt)
        w = (synth.make_uniform_logits((V, d), 400 + i) * (0.05 if bf16 else 1.0 / math.sqrt(d)))
        _check(h, w.to(dt), 2e-3 if bf16 else 2e-5, f"random-{i}")
