"""Category hidden expander and category-prior head: CPU oracle.

TEST INFRASTRUCTURE (see ``oracle/contract.py``): only tests, the smoke check and the benchmark's
CPU baseline use this module; the GPU library never does.

Sec. "Architecture": the trunk's hidden state h_k of every block position is mapped to R
category-specific branch states

    h_{k,z} = h_k + g_z(h_k),   g_z(h) = W_z h + c_z,

where the expander is a single linear layer from H to R*H (weight [R*H, H] in the nn.Linear
layout, output features ordered z-major: feature z*H + j is component j of g_z), and a separate
linear prior head maps the block-anchor hidden state to the category logits l = U h_anchor + e
(weight [R, H], bias [R]). The added parameter count is R H^2 + 2 R H + R (Table 4, with the
paper's K = R categories and hidden size H).

Arithmetic is binary64 on the given (bf16 or fp32) inputs; ``expand_branches`` can round the
result once to bf16 (round to nearest even), the type the branch states feed the head in.
"""
from __future__ import annotations

import numpy as np


def added_parameters(H: int, R: int) -> int:
    """Parameters of the expander (R*H*H weights + R*H biases) and prior head (R*H + R)."""
    return R * H * H + R * H + R * H + R


def expand_branches(h, W, c, round_bf16: bool = False):
    """Branch states h_{k,z} = h_k + W_z h_k + c_z.

    h [..., H] trunk states, W [R*H, H], c [R*H]. Returns [..., R, H] (binary64, or the bf16
    values as float64 when ``round_bf16``)."""
    h = np.asarray(h, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    c = np.asarray(c, dtype=np.float64)
    H = h.shape[-1]
    R = W.shape[0] // H
    g = h @ W.T + c                                        # [..., R*H], z-major features
    out = h[..., None, :] + g.reshape(h.shape[:-1] + (R, H))
    return bf16_round(out) if round_bf16 else out


def prior_logits(h_anchor, U, e):
    """Category logits l = U h_anchor + e; h_anchor [B, H], U [R, H], e [R] -> [B, R]."""
    return np.asarray(h_anchor, np.float64) @ np.asarray(U, np.float64).T + np.asarray(e, np.float64)


def bf16_round(x):
    """Round binary64 values to the nearest bfloat16 (8 significant bits, ties to even),
    returned as float64: x = m 2^E with 1/2 <= |m| < 1, and m 2^8 is rounded to an integer."""
    x = np.asarray(x, dtype=np.float64)
    m, E = np.frexp(x)
    return np.ldexp(np.rint(np.ldexp(m, 8)), E - 8)
