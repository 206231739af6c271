"""Determinism contract of the DBLast sampler and verifier: CPU oracle side.

TEST INFRASTRUCTURE. Only tests, the smoke check and the benchmark's CPU-baseline leg may
import anything under ``oracle/``. The product path never does.

The paper fixes *what* is sampled and accepted (the category draw and the per-position token
draws of the latent-mixture proposal, Sec. "Dependent Block Drafting and Verification"; the
accept probability min(1, p/q), Eq. accept-prob; the residual norm(max(p - q, 0)), Sec.
"Distributional correctness"). It is silent on how random numbers are produced and how a
floating-point probability becomes a discrete decision. This module fixes that reading so
that two independent implementations (this one and the HIP kernels) take every discrete
decision identically:

* every uniform draw is a word of Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random
  Numbers: As Easy as 1, 2, 3", SC'11), keyed by the seed and indexed by what it is for: word 0,
  and for the drafted token's second stage (the id within its 128-id tile) word 1 of the same
  counter;
* every probability that feeds a decision comes from a deterministic exponential built only
  from separately rounded IEEE add/sub/mul, round-to-nearest-even and exact power-of-two
  scaling (Cody-Waite range reduction followed by a Taylor polynomial in Horner form);
* every distribution that is sampled is quantised to unsigned integers at scale 2^40, so that
  its cumulative sums are exact and independent of summation order;
* inverse-CDF and accept decisions are exact integer comparisons.

Functions here are written for clarity, not speed.
"""
from __future__ import annotations

import math

import numpy as np

MASK32 = 0xFFFFFFFF

# Philox4x32 round multipliers and Weyl key increments (Salmon et al., SC'11, Sec. 5).
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
PHILOX_ROUNDS = 10

# Purposes: the second counter word says what a draw is for.
PURPOSE_CATEGORY = 0   # the latent category z of a block
PURPOSE_TOKEN = 1      # the drafted token at position k
PURPOSE_ACCEPT = 2     # the accept coin at position k
PURPOSE_RESIDUAL = 3   # the correction (residual) or bonus token

QSCALE_BITS = 40
QSCALE = float(2 ** QSCALE_BITS)


# ----------------------------------------------------------------------------------------
# Philox4x32-10
# ----------------------------------------------------------------------------------------
def philox4x32_10(ctr, key):
    """One Philox4x32-10 block on Python integers: 4 counter words, 2 key words -> 4 words.

    Each round multiplies counter words 0 and 2 by the two round constants, keeps the high
    and low halves of the 64-bit products, and mixes the high halves with the other counter
    words and the key; the key is advanced by the Weyl increments between rounds.
    """
    c0, c1, c2, c3 = (int(c) & MASK32 for c in ctr)
    k0, k1 = (int(k) & MASK32 for k in key)
    for _ in range(PHILOX_ROUNDS):
        p0 = PHILOX_M0 * c0
        p1 = PHILOX_M1 * c2
        hi0, lo0 = p0 >> 32, p0 & MASK32
        hi1, lo1 = p1 >> 32, p1 & MASK32
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0), lo1, (hi0 ^ c3 ^ k1), lo0
        k0 = (k0 + PHILOX_W0) & MASK32
        k1 = (k1 + PHILOX_W1) & MASK32
    return c0, c1, c2, c3


def philox4x32_10_np(c0, c1, c2, c3, k0, k1):
    """Vectorised Philox4x32-10 over numpy arrays (broadcast); words held in uint64."""
    u = np.uint64
    c0, c1, c2, c3, k0, k1 = np.broadcast_arrays(*(np.asarray(a, dtype=np.uint64) & u(MASK32)
                                                   for a in (c0, c1, c2, c3, k0, k1)))
    c0, c1, c2, c3, k0, k1 = (a.copy() for a in (c0, c1, c2, c3, k0, k1))
    m32 = u(MASK32)
    for _ in range(PHILOX_ROUNDS):
        p0 = u(PHILOX_M0) * c0
        p1 = u(PHILOX_M1) * c2
        hi0, lo0 = p0 >> u(32), p0 & m32
        hi1, lo1 = p1 >> u(32), p1 & m32
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0), lo1, (hi0 ^ c3 ^ k1), lo0
        k0 = (k0 + u(PHILOX_W0)) & m32
        k1 = (k1 + u(PHILOX_W1)) & m32
    return c0, c1, c2, c3


def draw_u32(seed: int, purpose: int, k: int, seq: int, step: int) -> int:
    """The uniform 32-bit word for (purpose, position k, sequence seq, step) under seed.

    counter = (k, purpose, seq mod 2^32, step mod 2^32), key = (seed low word, seed high word);
    the draw is output word 0.
    """
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return philox4x32_10((k, purpose, seq, step), (seed & MASK32, seed >> 32))[0]


def draw_u32_word1(seed: int, purpose: int, k: int, seq: int, step: int) -> int:
    """Output word 1 of the same Philox block as ``draw_u32`` (the drafted token's id within
    the tile that word 0 selected)."""
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return philox4x32_10((k, purpose, seq, step), (seed & MASK32, seed >> 32))[1]


class PhiloxDraws:
    """Supplies draws for one block (fixed seed, sequence index and step)."""

    def __init__(self, seed: int, seq: int, step: int):
        self.seed, self.seq, self.step = int(seed), int(seq), int(step)

    def __call__(self, purpose: int, k: int) -> int:
        return draw_u32(self.seed, purpose, k, self.seq, self.step)


# ----------------------------------------------------------------------------------------
# Deterministic exponentials
# ----------------------------------------------------------------------------------------
_F = np.float32
# 1/ln 2 rounded to binary32 (bits 0x3FB8AA3B).
LOG2E_F32 = _F(1.4426950408889634)
# ln 2 cut to 15 significant bits, so that n * LN2_HI_F32 is exact for |n| <= 128.
LN2_HI_F32 = _F(0.693145751953125)
# The rest of ln 2, rounded to binary32 (bits 0x35BFBE8E).
LN2_LO_F32 = _F(1.428606765330187e-06)
# Taylor coefficients 1/j!, j = 0..7, each the binary32 rounding of the binary64 value.
EXP_COEF_F32 = [_F(1.0 / math.factorial(j)) for j in range(8)]
EXP_CUTOFF_F32 = _F(-80.0)

# binary64 twins: ln 2 rounded to 32 significant bits (exact products for |n| < 2^21).
LOG2E_F64 = 1.4426950408889634
LN2_HI_F64 = float.fromhex("0x1.62e42ff000000p-1")
LN2_LO_F64 = float.fromhex("-0x1.718432a1b0e26p-35")
EXP_COEF_F64 = [1.0 / math.factorial(j) for j in range(14)]
EXP_CUTOFF_F64 = -708.0


def detexp32(x):
    """Deterministic binary32 e^x for the sampling and accept decisions.

    Inputs above 0 are clamped to 0 (log-probabilities), inputs below -80, -inf and NaN give 0.
    Otherwise n = rint(x log2 e), r = (x - n ln2_hi) - n ln2_lo, e^r by a degree-7 Taylor
    polynomial in Horner form, and the result is scaled by 2^n. Every operation is a separately
    rounded binary32 operation.
    """
    x = np.asarray(x, dtype=np.float32)
    valid = x > EXP_CUTOFF_F32
    xc = np.where(valid, np.minimum(x, _F(0.0)), _F(0.0)).astype(np.float32)
    n = np.rint(xc * LOG2E_F32).astype(np.float32)
    r = ((xc - n * LN2_HI_F32) - n * LN2_LO_F32).astype(np.float32)
    p = np.full_like(r, EXP_COEF_F32[7])
    for j in range(6, -1, -1):
        p = (p * r).astype(np.float32)
        p = (p + EXP_COEF_F32[j]).astype(np.float32)
    y = np.ldexp(p, n.astype(np.int32)).astype(np.float32)
    return np.where(valid, y, _F(0.0)).astype(np.float32)


def dexp64(x):
    """Deterministic binary64 e^x (same recipe, degree-13 polynomial, cut-off -708)."""
    x = np.asarray(x, dtype=np.float64)
    valid = x > EXP_CUTOFF_F64
    xc = np.where(valid, np.minimum(x, 0.0), 0.0)
    n = np.rint(xc * LOG2E_F64)
    r = (xc - n * LN2_HI_F64) - n * LN2_LO_F64
    p = np.full_like(r, EXP_COEF_F64[13])
    for j in range(12, -1, -1):
        p = p * r
        p = p + EXP_COEF_F64[j]
    y = np.ldexp(p, n.astype(np.int32))
    return np.where(valid, y, 0.0)


# ----------------------------------------------------------------------------------------
# Fixed-point quantisation and integer decisions
# ----------------------------------------------------------------------------------------
def quant40(y):
    """floor(y * 2^40) as uint64 for binary32 or binary64 y in [0, 1]."""
    y = np.asarray(y)
    return np.floor(y.astype(np.float64) * QSCALE).astype(np.uint64)


def icdf(weights, r: int) -> int:
    """Inverse CDF on integer weights with a 32-bit uniform word r.

    Z = sum of the weights, T = floor(r * Z / 2^32); the result is the smallest index i whose
    inclusive cumulative sum exceeds T, so zero-weight entries are never chosen. Returns -1
    when Z = 0.
    """
    w = np.asarray(weights, dtype=np.uint64)
    cum = np.cumsum(w, dtype=np.uint64)
    Z = int(cum[-1]) if cum.size else 0
    if Z == 0:
        return -1
    T = (int(r) * Z) >> 32
    return int(np.searchsorted(cum, np.uint64(T), side="right"))


def accept_int(r: int, q_int: int, p_int: int) -> bool:
    """Exact integer form of u < p/q with u = r / 2^32: r * q_int < p_int * 2^32."""
    return int(r) * int(q_int) < (int(p_int) << 32)
