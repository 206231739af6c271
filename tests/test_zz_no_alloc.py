"""dbl_verify_block_static (the allocation-free verification entry point, for callers that
cannot allocate) against dbl_verify_block on the same inputs, through the C ABI: two calls in a
row, the second with a smaller batch, each bit-identical to the workspace entry point (tokens,
acceptance masses, AL_b and E)."""
import pytest
import torch

from cases import BlockCase

pytestmark = pytest.mark.gpu


def _both(D, c, seed, step, so):
    tls, lmass, lse, ell, logp = c.device()
    _, x = D.dbl_sample_block(tls, lmass, lse, ell, seed=seed, step=step, seq_offset=so)
    ref = D.dbl_verify_block(tls, lmass, lse, ell, x, logp, seed=seed, step=step, seq_offset=so)
    got = D.dbl_verify_block_static(tls, lmass, lse, ell, x, logp, seed=seed, step=step,
                                    seq_offset=so)
    torch.cuda.synchronize()
    return ref, got


def test_static_scratch_verify_matches_workspace_verify_twice():
    from paper_2608_05448_amd import dblast as D
    big = BlockCase(64, 8, 8, 3000, d=16, seed=71, target="aligned-block", noise=0.1)
    small = BlockCase(5, 6, 3, 1001, d=16, seed=72, target="aligned", kp_extra=0)
    for name, c, so in (("B=64 K=8 R=8 V=3000", big, 0), ("B=5 K=6 R=3 V=1001", small, 9)):
        print(f"[no-alloc] {name}", flush=True)
        ref, got = _both(D, c, seed=5, step=2, so=so)
        for k in ("n_accept", "next_token", "accept_mass", "al_expected", "exp_len"):
            assert torch.equal(ref[k], got[k]), k
        na = got["n_accept"].cpu().numpy()
        print(f"[no-alloc] {name}: n_accept {na.tolist()[:12]}", flush=True)
