"""GPU parity of dbl_acceptance_objective against the oracle (Eqs. dependent-nll,
acceptance-length-objective, subblock-objective).

Both sides read the same branch log-probabilities (the oracle head's output on synthetic
inputs), category logits, target log-probabilities and trajectories (drawn from the target with a
seeded generator). Real-valued outputs agree to binary64 rounding of binary32 inputs (checked at
1e-5); l_tau must match exactly unless the oracle's log r at the deciding position lies within
1e-9 of log tau (a certified near-tie of the binary64 comparison).
"""
import zlib

import numpy as np
import pytest
import torch

from cases import BlockCase
from oracle import objective as OB

pytestmark = pytest.mark.gpu

CASES = [
    # name, B, K, R, V, d, target, T, z_temp, tau
    ("aligned", 16, 8, 4, 2000, 16, "aligned", 1.0, 1.0, 0.1),
    ("independent", 16, 8, 4, 2000, 16, "independent", 1.0, 1.0, 0.1),
    ("single-category", 12, 10, 1, 700, 16, "aligned", 0.7, 1.0, 0.1),
    ("max-categories", 4, 6, 64, 500, 16, "aligned", 1.0, 1.0, 0.1),
    ("zero-cat-temp", 8, 6, 5, 1000, 16, "aligned", 1.0, 0.0, 0.1),
    ("long-block", 4, 40, 8, 300, 8, "aligned", 1.0, 1.0, 0.05),
    ("loose-tau", 16, 8, 4, 1001, 16, "aligned", 1.5, 0.8, 0.9),
    ("tight-tau", 16, 8, 4, 1001, 16, "aligned", 1.0, 1.2, 1e-4),
]


def _close(got, want, tol=1e-5):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    fin = np.isfinite(want)
    assert np.array_equal(np.isfinite(got), fin)
    err = np.abs(got[fin] - want[fin]) / np.maximum(1.0, np.abs(want[fin]))
    assert err.size == 0 or err.max() < tol, err.max()


def _objective_case(name, B, K, R, V, d, target, T, zt, tau, seed):
    """One objective call at this shape against the oracle (trajectories drawn from the target)."""
    from paper_2608_05448_amd import dblast as D
    print(f"[objective] {name} B={B} K={K} R={R} V={V} T={T} z_temp={zt} tau={tau}", flush=True)
    c = BlockCase(B, K, R, V, d=d, seed=seed % 1000, target=target, kp_extra=0, T=T)
    rng = np.random.default_rng(seed)
    p = np.exp(c.logp.astype(np.float64))
    cum = np.cumsum(p / p.sum(-1, keepdims=True), axis=-1)
    xs = np.minimum((cum < rng.random((B, K, 1))).sum(-1), V - 1).astype(np.int32)
    tls, lmass, lse, ell, logp = c.device()
    out = D.dbl_acceptance_objective(tls, lmass, lse, ell, torch.from_numpy(xs).cuda(), logp,
                                     z_temp=zt, tau=tau)
    torch.cuda.synchronize()
    ref = OB.acceptance_objective(c.lq, c.ell, zt, xs, c.logp, tau=tau)
    _close(out["log_r"].cpu().numpy(), ref["log_r"])
    _close(out["S"].cpu().numpy(), ref["S"])
    _close(out["nll"].cpu().numpy(), ref["nll"])
    lt = out["ell_tau"].cpu().numpy()
    same = lt == ref["ell_tau"]
    for b in np.nonzero(~same)[0]:
        l = min(lt[b], ref["ell_tau"][b])
        assert abs(ref["log_r"][b, l - 1] - np.log(tau)) < 1e-9, (b, lt[b], ref["ell_tau"][b])
    _close(out["J"].cpu().numpy()[same], ref["J"][same], tol=1e-4)
    print(f"[objective] {name}: mean l_tau {lt.mean():.2f}, mean J {ref['J'].mean():.3f}",
          flush=True)
    if R == 1:   # Eq. independent-nll: the sum of per-position cross-entropies
        ce = -np.sum(c.lq[np.arange(B)[:, None], np.arange(K)[None, :], 0, xs], axis=1)
        _close(out["nll"].cpu().numpy(), ce)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_objective_parity(case):
    _objective_case(*case, zlib.crc32(case[0].encode()))


def test_objective_random_shapes():
    """A seeded sweep of random small shapes (K = 1 included, V below one tile, odd R, target
    temperature 0, a range of tau) against the oracle."""
    rng = np.random.default_rng(20261205)
    for i in range(12):
        B, K, R = int(rng.integers(1, 20)), int(rng.integers(1, 24)), int(rng.integers(1, 20))
        V = int(rng.choice([int(rng.integers(2, 128)), int(rng.integers(128, 4000))]))
        target = str(rng.choice(["aligned", "independent"]))
        T = float(rng.choice([0.0, 0.7, 1.0, 1.5]))
        zt = float(rng.choice([0.0, 0.5, 1.0, 2.0]))
        tau = float(rng.choice([1e-4, 0.05, 0.1, 0.5, 0.9]))
        _objective_case(f"random-{i}", B, K, R, V, 8, target, T, zt, tau, 500 + i)
