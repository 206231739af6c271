"""GPU parity of dbl_sample_block, dbl_verify_block and dbl_expected_len against the oracle.

Both sides receive the same branch log-probabilities (the oracle head's output on synthetic
inputs), category logits and target log-probabilities. Token indices (category, drafted
tokens, accepted count, residual/bonus token) must match bit for bit; acceptance masses,
AL_b and E within 1e-4 relative.
"""
import zlib

import numpy as np
import pytest
import torch

from cases import BlockCase
from oracle import mixture as MX

pytestmark = pytest.mark.gpu

CASES = [
    # name, B, K, R, V, d, target, kp_extra, T, z_temp, seed, step, seq_offset
    ("aligned-bonus", 6, 5, 3, 3000, 32, "aligned", 1, 1.0, 1.0, 0, 0, 0),
    ("independent", 6, 5, 3, 3000, 32, "independent", 0, 1.0, 1.0, 1, 3, 17),
    ("zero-cat-temp", 5, 4, 4, 1000, 16, "aligned", 1, 0.7, 0.0, 2, 1, 0),
    ("single-category", 8, 6, 1, 700, 16, "aligned", 1, 1.0, 1.0, 3, 0, 5),
    ("full-vocab", 2, 3, 4, 151936, 16, "aligned", 1, 1.0, 0.8, 2**40 + 5, 7, 1000),
    ("tiny-vocab", 3, 4, 2, 77, 8, "aligned", 1, 1.0, 1.5, 4, 2, 0),
    ("max-categories", 2, 3, 64, 500, 16, "aligned", 0, 1.0, 1.0, 5, 0, 9),
    ("greedy-target", 4, 5, 3, 900, 16, "aligned", 1, 0.0, 1.0, 6, 0, 0),
    ("many-blocks", 64, 4, 2, 1000, 16, "aligned", 1, 1.0, 1.0, 7, 11, 123456),
    ("ragged-vocab", 3, 4, 3, 1001, 16, "aligned", 1, 0.6, 1.0, 8, 0, 0),
    ("long-block", 2, 40, 64, 300, 8, "aligned", 1, 1.0, 1.0, 9, 0, 0),   # K*R > 2048
    ("wide-categories", 3, 6, 5, 2000, 16, "aligned", 1, 1.0, 2.0, 10, 5, 3),  # R not 1,2,4,8,16
    # The verification kernels the benchmark times are specialised on R: R = 8 (Qwen3 step
    # workloads) and R = 16 (objective workload), here with the bonus row.
    ("bench-variant-r8", 128, 8, 8, 2000, 16, "aligned-block", 1, 1.0, 1.0, 11, 2, 40),
    ("objective-variant-r16", 96, 6, 16, 1500, 16, "aligned-block", 1, 1.0, 1.0, 12, 0, 7),
    ("r4-stress-variant", 96, 8, 4, 1200, 16, "aligned-block", 1, 1.0, 1.0, 13, 999, 0),
    # K > 64: the parallel chain takes its accept decisions in two 64-position rounds.
    ("long-chain", 3, 100, 2, 500, 8, "aligned-block", 1, 1.0, 1.0, 14, 0, 0),
    # K > 256: sequential chain, and the finalize kernel carries E across position chunks.
    ("chunked-finalize", 2, 300, 1, 300, 8, "aligned-block", 1, 1.0, 1.0, 15, 1, 3),
    # 256 < K R <= 2048: the parallel chain gathers in a loop; 17 <= R <= 32 normalises over
    # 32-lane segments, R <= 16 over 8-lane segments.
    ("looped-gather-r24", 4, 12, 24, 800, 16, "aligned-block", 1, 1.0, 1.0, 16, 0, 2),
    ("looped-gather-r8", 16, 40, 8, 600, 16, "aligned-block", 1, 1.0, 1.0, 17, 4, 0),
    # More than 2048 tiles per row: the workgroup inverse CDFs walk runs of 10 tile sums or masses
    # instead of holding them in registers.
    ("huge-vocab", 3, 3, 2, 300000, 8, "aligned", 1, 1.0, 1.0, 18, 0, 0),
]
NOISE = {"bench-variant-r8": 0.1, "objective-variant-r16": 0.1, "r4-stress-variant": 0.1,
         "long-chain": 0.02, "chunked-finalize": 0.02, "looped-gather-r24": 0.05,
         "looped-gather-r8": 0.02}


def _rel_close(got, want, rtol=1e-4, floor=1e-30):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    mask = np.abs(want) > floor
    if mask.any():
        rel = np.max(np.abs(got[mask] - want[mask]) / np.abs(want[mask]))
        assert rel < rtol, rel
    assert np.all(np.abs(got[~mask]) < 1e-20)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_sample_verify_parity(case):
    from paper_2608_05448_amd import dblast as D
    name, B, K, R, V, d, target, kx, T, zt, seed, step, so = case
    print(f"[sample/verify] {name} B={B} K={K} R={R} V={V} seed={seed} step={step}", flush=True)
    c = BlockCase(B, K, R, V, d=d, seed=zlib.crc32(name.encode()) % 1000, target=target, kp_extra=kx, T=T,
                  noise=NOISE.get(name, 0.3))
    tls, lmass, lse, ell, logp = c.device()
    seq = so + np.arange(B)

    z_g, x_g = D.dbl_sample_block(tls, lmass, lse, ell, z_temp=zt, seed=seed, step=step,
                                  seq_offset=so)
    torch.cuda.synchronize()
    z_o, x_o = MX.sample_blocks(c.tls, c.lmass, c.lse, c.ell, zt, seed, step, seq)
    np.testing.assert_array_equal(z_g.cpu().numpy(), z_o)
    np.testing.assert_array_equal(x_g.cpu().numpy(), x_o)

    out = D.dbl_verify_block(tls, lmass, lse, ell, x_g, logp, z_temp=zt, seed=seed, step=step,
                             seq_offset=so)
    torch.cuda.synchronize()
    ref = MX.verify_blocks(c.lq, c.ell, zt, x_o, c.logp, seed, step, seq)
    na = out["n_accept"].cpu().numpy()
    print(f"[sample/verify] {name} n_accept={na.tolist()[:16]}", flush=True)
    np.testing.assert_array_equal(na, ref["n_accept"])
    np.testing.assert_array_equal(out["next_token"].cpu().numpy(), ref["next_token"])
    _rel_close(out["accept_mass"].cpu().numpy(), ref["beta"])
    _rel_close(out["al_expected"].cpu().numpy(), ref["al"])
    _rel_close(out["exp_len"].cpu().numpy(), ref["E"])

    # Expected length along a different (target-side) trajectory.
    rng = np.random.default_rng(seed % 2**32)
    xs = rng.integers(0, V, size=(B, K)).astype(np.int32)
    beta_g, e_g = D.dbl_expected_len(tls, lmass, lse, ell, torch.from_numpy(xs).cuda(),
                                     logp[:, :K].contiguous(), z_temp=zt)
    torch.cuda.synchronize()
    beta_o, e_o = MX.expected_len_blocks(c.lq, c.ell, zt, xs, c.logp[:, :K])
    _rel_close(beta_g.cpu().numpy(), beta_o)
    _rel_close(e_g.cpu().numpy(), e_o)


def test_accept_paths_are_exercised():
    """The aligned cases reach accepts, rejections with a residual and full acceptance."""
    from paper_2608_05448_amd import dblast as D
    c = BlockCase(64, 4, 2, 400, d=16, seed=99, target="aligned", kp_extra=1, q_sharp=0.5)
    tls, lmass, lse, ell, logp = c.device()
    _, x = D.dbl_sample_block(tls, lmass, lse, ell, seed=1)
    out = D.dbl_verify_block(tls, lmass, lse, ell, x, logp, seed=1)
    torch.cuda.synchronize()
    na = out["n_accept"].cpu().numpy()
    ref = MX.verify_blocks(c.lq, c.ell, 1.0, x.cpu().numpy(), c.logp, 1, 0, np.arange(64))
    np.testing.assert_array_equal(na, ref["n_accept"])
    np.testing.assert_array_equal(out["next_token"].cpu().numpy(), ref["next_token"])
    assert (na == 0).any() and ((na > 0) & (na < 4)).any() and (na == 4).any(), na


def test_stream_several_chunks_per_workgroup():
    """R = 4 with a grid large enough that each stream workgroup takes several 32-tile chunks
    (256 blocks, 8 position rows, 5 chunks of which the last is partial, all in one workgroup):
    every output against the oracle, with all accept paths."""
    from paper_2608_05448_amd import dblast as D
    B, K, R, V = 256, 7, 4, 20000
    print(f"[sample/verify] several chunks per workgroup R={R} K={K} B={B} V={V}", flush=True)
    c = BlockCase(B, K, R, V, d=16, seed=77, target="aligned-block", kp_extra=1, noise=0.1)
    tls, lmass, lse, ell, logp = c.device()
    seq = np.arange(B)
    z, x = D.dbl_sample_block(tls, lmass, lse, ell, seed=5, step=2)
    out = D.dbl_verify_block(tls, lmass, lse, ell, x, logp, seed=5, step=2)
    torch.cuda.synchronize()
    z_o, x_o = MX.sample_blocks(c.tls, c.lmass, c.lse, c.ell, 1.0, 5, 2, seq)
    np.testing.assert_array_equal(z.cpu().numpy(), z_o)
    np.testing.assert_array_equal(x.cpu().numpy(), x_o)
    ref = MX.verify_blocks(c.lq, c.ell, 1.0, x_o, c.logp, 5, 2, seq)
    na = out["n_accept"].cpu().numpy()
    np.testing.assert_array_equal(na, ref["n_accept"])
    np.testing.assert_array_equal(out["next_token"].cpu().numpy(), ref["next_token"])
    _rel_close(out["accept_mass"].cpu().numpy(), ref["beta"])
    _rel_close(out["al_expected"].cpu().numpy(), ref["al"])
    _rel_close(out["exp_len"].cpu().numpy(), ref["E"])
    counts = ((na == 0).sum(), ((na > 0) & (na < K)).sum(), (na == K).sum())
    print(f"[sample/verify] several chunks: reject at 0 / after accepts / full: {counts}", flush=True)
    assert all(n > 0 for n in counts), counts


@pytest.mark.parametrize("R,K", [(8, 8), (16, 6), (4, 8)])
def test_accept_paths_at_the_benchmark_variants(R, K):
    """R = 8 / 16 / 4 (the specialisations the Qwen3, objective and stress workloads run):
    rejection at the first position, rejection after accepts (residual at k > 0) and full
    acceptance with a bonus token all occur, and every output matches the oracle."""
    from paper_2608_05448_amd import dblast as D
    B, V = 256, 2000
    print(f"[sample/verify] accept paths R={R} K={K} B={B} V={V}", flush=True)
    c = BlockCase(B, K, R, V, d=16, seed=40 + R, target="aligned-block", kp_extra=1, noise=0.1)
    tls, lmass, lse, ell, logp = c.device()
    seq = np.arange(B)
    z, x = D.dbl_sample_block(tls, lmass, lse, ell, seed=3, step=1)
    out = D.dbl_verify_block(tls, lmass, lse, ell, x, logp, seed=3, step=1)
    torch.cuda.synchronize()
    z_o, x_o = MX.sample_blocks(c.tls, c.lmass, c.lse, c.ell, 1.0, 3, 1, seq)
    np.testing.assert_array_equal(z.cpu().numpy(), z_o)
    np.testing.assert_array_equal(x.cpu().numpy(), x_o)
    ref = MX.verify_blocks(c.lq, c.ell, 1.0, x_o, c.logp, 3, 1, seq)
    na = out["n_accept"].cpu().numpy()
    np.testing.assert_array_equal(na, ref["n_accept"])
    np.testing.assert_array_equal(out["next_token"].cpu().numpy(), ref["next_token"])
    _rel_close(out["accept_mass"].cpu().numpy(), ref["beta"])
    _rel_close(out["al_expected"].cpu().numpy(), ref["al"])
    _rel_close(out["exp_len"].cpu().numpy(), ref["E"])
    counts = ((na == 0).sum(), ((na > 0) & (na < K)).sum(), (na == K).sum())
    print(f"[sample/verify] R={R}: reject at 0 / after accepts / full: {counts}", flush=True)
    assert all(n > 0 for n in counts), counts
    assert np.all(out["next_token"].cpu().numpy()[na == K] >= 0)   # bonus drawn


def test_repeated_calls_are_bit_identical():
    from paper_2608_05448_amd import dblast as D
    c = BlockCase(4, 5, 3, 2000, d=16, seed=5)
    tls, lmass, lse, ell, logp = c.device()
    runs = []
    for _ in range(3):
        z, x = D.dbl_sample_block(tls, lmass, lse, ell, seed=42, step=3)
        o = D.dbl_verify_block(tls, lmass, lse, ell, x, logp, seed=42, step=3)
        torch.cuda.synchronize()
        runs.append([t.cpu().numpy().tobytes() for t in (z, x, o["n_accept"], o["next_token"],
                                                          o["accept_mass"], o["exp_len"])])
    assert runs[0] == runs[1] == runs[2]


def test_out_of_range_draft_ids_are_rejected_without_faulting():
    from paper_2608_05448_amd import dblast as D
    c = BlockCase(3, 4, 2, 300, d=16, seed=6)
    tls, lmass, lse, ell, logp = c.device()
    x = torch.tensor([[-1, 5, 6, 7], [300, 1, 2, 3], [4, 5, 2**30, 7]], dtype=torch.int32,
                     device="cuda")
    o = D.dbl_verify_block(tls, lmass, lse, ell, x, logp, seed=0)
    torch.cuda.synchronize()
    na = o["n_accept"].cpu().numpy()
    assert na[0] == 0 and na[1] == 0 and na[2] <= 2
    assert np.all(o["al_expected"].cpu().numpy()[:2] == 0.0)


def test_random_shapes_against_the_oracle():
    """A seeded sweep of small random shapes (B, K, R, V, Kp, target, temperatures), so that
    combinations the cases above do not name (K = 1, V below one tile, odd R, ragged last tiles,
    with and without the bonus row) go through the draw, the verification and the
    expected-length reduction against the oracle."""
    from paper_2608_05448_amd import dblast as D
    rng = np.random.default_rng(20261202)
    for i in range(14):
        B = int(rng.integers(1, 24))
        K = int(rng.integers(1, 20))
        R = int(rng.integers(1, 20))
        V = int(rng.choice([int(rng.integers(1, 128)), int(rng.integers(128, 6000))]))
        kx = int(rng.integers(0, 2))
        target = str(rng.choice(["aligned", "aligned-block", "independent"]))
        zt = float(rng.choice([0.0, 0.5, 1.0, 2.0]))
        T = float(rng.choice([0.0, 0.7, 1.0]))
        seed, step, so = int(rng.integers(0, 2**40)), int(rng.integers(0, 1000)), int(rng.integers(0, 999))
        print(f"[random] {i}: B={B} K={K} R={R} V={V} Kp=K+{kx} {target} z_temp={zt} T={T} "
              f"seed={seed} step={step} so={so}", flush=True)
        c = BlockCase(B, K, R, V, d=8, seed=100 + i, target=target, kp_extra=kx, T=T, noise=0.05)
        tls, lmass, lse, ell, logp = c.device()
        seq = so + np.arange(B)
        z, x = D.dbl_sample_block(tls, lmass, lse, ell, z_temp=zt, seed=seed, step=step,
                                  seq_offset=so)
        out = D.dbl_verify_block(tls, lmass, lse, ell, x, logp, z_temp=zt, seed=seed, step=step,
                                 seq_offset=so)
        torch.cuda.synchronize()
        z_o, x_o = MX.sample_blocks(c.tls, c.lmass, c.lse, c.ell, zt, seed, step, seq)
        np.testing.assert_array_equal(z.cpu().numpy(), z_o)
        np.testing.assert_array_equal(x.cpu().numpy(), x_o)
        ref = MX.verify_blocks(c.lq, c.ell, zt, x_o, c.logp, seed, step, seq)
        np.testing.assert_array_equal(out["n_accept"].cpu().numpy(), ref["n_accept"])
        np.testing.assert_array_equal(out["next_token"].cpu().numpy(), ref["next_token"])
        _rel_close(out["accept_mass"].cpu().numpy(), ref["beta"])
        _rel_close(out["al_expected"].cpu().numpy(), ref["al"])
        _rel_close(out["exp_len"].cpu().numpy(), ref["E"])
        # The expected-length reduction along a random trajectory of the same shape.
        xs = rng.integers(0, V, size=(B, K)).astype(np.int32)
        beta_g, e_g = D.dbl_expected_len(tls, lmass, lse, ell, torch.from_numpy(xs).cuda(),
                                         logp[:, :K].contiguous(), z_temp=zt)
        torch.cuda.synchronize()
        beta_o, e_o = MX.expected_len_blocks(c.lq, c.ell, zt, xs, c.logp[:, :K])
        _rel_close(beta_g.cpu().numpy(), beta_o)
        _rel_close(e_g.cpu().numpy(), e_o)
