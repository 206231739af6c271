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
                 q_sharp=2.0, noise=0.3):
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
        if target in ("aligned", "aligned-block"):
            # "aligned": the target at position k follows branch (b + k) % R of the drafter,
            # plus noise, so most drafted tokens have comparable p and q. "aligned-block": every
            # position of block b follows branch b % R, so blocks whose drawn category is b % R
            # are often accepted in full (and the bonus row is drawn from).
            base = torch.from_numpy(self.lq.astype(np.float64))
            shift = torch.arange(K)[None, :] if target == "aligned" else 0 * torch.arange(K)[None, :]
            idx = (torch.arange(B)[:, None] + shift) % R
            follow = base[torch.arange(B)[:, None], torch.arange(K)[None, :], idx]
            g[:, :K] = follow + noise * g[:, :K]
        self.logp = synth.target_logprobs(g, T).numpy()

    def device(self):
        dev = "cuda"
        f = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        return f(self.tls), f(self.lmass), f(self.lse), f(self.ell), f(self.logp)


_ORACLE_FULL: dict = {}


def _oracle_full(name: str, h: torch.Tensor, w: torch.Tensor):
    if name not in _ORACLE_FULL:
        _ORACLE_FULL.clear()
        d = h.shape[-1]
        tls, lmass, lse = OH.head_factored(np32(h).reshape(-1, d), np32(w), v_chunk=8192)
        _ORACLE_FULL[name] = (tls, lmass, lse, OH.flat_logq(tls, lmass, lse))
    return _ORACLE_FULL[name]


def oracle_full_head(name: str, h: torch.Tensor, w: torch.Tensor) -> np.ndarray:
    """The oracle's branch log-probs [M, V] (binary32 flat form) for a whole workload's head,
    from the exact inputs h [B, K, R, d] and w [V, d] the GPU consumed (binary64 GEMM and
    log-softmax). Computed once per process for the most recent workload name."""
    return _oracle_full(name, h, w)[3]


def oracle_full_factored(name: str, h: torch.Tensor, w: torch.Tensor):
    """The same head in its binary32 two-level form (tls [M, V], lmass [M, nT], lse [M])."""
    return _oracle_full(name, h, w)[:3]
