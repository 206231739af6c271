"""Test inputs built from the seeded generators (synth) and the CPU oracle only.

Nothing here reads a value produced by the HIP library: the GPU and the oracle receive the
same bytes, and expected values come from the oracle.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import synth
from oracle import head as OH


def np32(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float32).numpy()


def flat_from_factored(tls, lmass, lse):
    """fl32(tls + fl32(lmass - lse)) in numpy for arrays [..., V], [..., nT], [...]."""
    tls, lmass, lse = (np.asarray(a, np.float32) for a in (tls, lmass, lse))
    off = (lmass - lse[..., None]).astype(np.float32)
    return (tls + np.repeat(off, 128, axis=-1)[..., :tls.shape[-1]]).astype(np.float32)


class BlockCase:
    """Branch log-probs (oracle head on synthetic h, w), category logits and a target."""

    def __init__(self, B, K, R, V, d=32, seed=0, target="aligned", kp_extra=1, T=1.0,
                 q_sharp=2.0):
        self.B, self.K, self.R, self.V, self.d = B, K, R, V, d
        h = synth.make_uniform_logits((B * K * R, d), seed * 7 + 1).to(torch.float32)
        w = synth.make_uniform_logits((V, d), seed * 7 + 2, scale=q_sharp / math.sqrt(d))
        w = w.to(torch.float32)
        tls, lmass, lse = OH.head_factored(h.numpy(), w.numpy())
        nT = OH.n_tiles(V)
        self.tls = tls.reshape(B, K, R, V)
        self.lmass = lmass.reshape(B, K, R, nT)
        self.lse = lse.reshape(B, K, R)
        self.lq = flat_from_factored(self.tls, self.lmass, self.lse)
        self.ell = synth.make_uniform_logits((B, R), seed * 7 + 3).to(torch.float32).numpy()
        Kp = K + kp_extra
        g = synth.make_uniform_logits((B, Kp, V), seed * 7 + 4, scale=2.0)
        if target == "aligned":
            # The target at position k follows branch (b + k) % R of the drafter, plus noise:
            # most drafted tokens then have comparable p and q and the accept path is exercised.
            base = torch.from_numpy(self.lq.astype(np.float64))
            idx = (torch.arange(B)[:, None] + torch.arange(K)[None, :]) % R
            follow = base[torch.arange(B)[:, None], torch.arange(K)[None, :], idx]
            g[:, :K] = follow + 0.3 * g[:, :K]
        self.logp = synth.target_logprobs(g, T).numpy()

    def device(self):
        dev = "cuda"
        f = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        return f(self.tls), f(self.lmass), f(self.lse), f(self.ell), f(self.logp)
