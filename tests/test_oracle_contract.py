"""Pins of the determinism contract (CPU oracle): Philox, exponentials, integer decisions."""
import math
import os
import struct
from fractions import Fraction

import numpy as np
import pytest

from oracle import contract as C
from oracle import mixture as MX

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _kat():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                rows.append([int(t, 16) for t in line.split()])
    return rows


def test_philox_known_answers():
    rows = _kat()
    assert len(rows) == 3
    for r in rows:
        ctr, key, want = r[0:4], r[4:6], r[6:10]
        assert list(C.philox4x32_10(ctr, key)) == want


def test_philox_vectorised_matches_scalar():
    rng = np.random.default_rng(7)
    words = rng.integers(0, 2**32, size=(200, 6), dtype=np.uint64)
    got = C.philox4x32_10_np(*[words[:, i] for i in range(6)])
    for i in range(words.shape[0]):
        w = [int(v) for v in words[i]]
        assert tuple(int(g[i]) for g in got) == C.philox4x32_10(w[0:4], w[4:6])


def test_batched_draws_match_scalar_draws():
    seed = (0xDEADBEEF << 32) | 0x12345678
    seqs = np.array([0, 1, 5, 2**32 + 3, 77], dtype=np.uint64)
    for purpose in range(4):
        for k in (0, 3, 15):
            got = MX.draws(seed, purpose, k, seqs, 11)
            want = [C.draw_u32(seed, purpose, k, int(s), 11) for s in seqs]
            assert [int(g) for g in got] == want


def _bits32(x):
    return struct.unpack("<I", struct.pack("<f", float(x)))[0]


def test_exp_constants_have_documented_bits():
    # The HIP side writes these constants as literals; these are the values both must hold.
    assert _bits32(C.LOG2E_F32) == 0x3FB8AA3B
    assert _bits32(C.LN2_HI_F32) == 0x3F317200
    assert _bits32(C.LN2_LO_F32) == 0x35BFBE8E
    assert C.LN2_HI_F64.hex() == "0x1.62e42ff000000p-1"
    assert C.LN2_LO_F64.hex() == "-0x1.718432a1b0e26p-35"
    # n * ln2_hi must be exact over the whole reduced range.
    for n in range(-130, 1):
        assert float(np.float32(n) * C.LN2_HI_F32) == n * float(C.LN2_HI_F32)
    for n in range(-1100, 1):
        assert Fraction(n * C.LN2_HI_F64) == n * Fraction(C.LN2_HI_F64)
    # hi + lo approximates ln 2 to far better than binary32 / binary64 precision.
    ln2 = Fraction("0.693147180559945309417232121458176568075500134360255254120680")
    assert abs(Fraction(float(C.LN2_HI_F32)) + Fraction(float(C.LN2_LO_F32)) - ln2) <= Fraction(1, 2**44)
    assert abs(Fraction(C.LN2_HI_F64) + Fraction(C.LN2_LO_F64) - ln2) < Fraction(1, 2**85)


def test_detexp32_accuracy_and_special_values():
    x = np.linspace(-79.99, 0.0, 400001, dtype=np.float32)
    y = C.detexp32(x).astype(np.float64)
    ref = np.exp(x.astype(np.float64))
    ulp = np.spacing(ref.astype(np.float32)).astype(np.float64)
    assert np.max(np.abs(y - ref) / ulp) <= 2.0
    sp = C.detexp32(np.array([0.0, -0.0, 1.0, 50.0, -80.0, -np.inf, np.nan], dtype=np.float32))
    assert list(sp) == [1.0, 1.0, 1.0, 1.0, 0.0, 0.0, 0.0]
    # Exact powers of two from exact multiples of ln 2 are not expected, but monotonic non-
    # decreasing behaviour over a fine grid is: a sign error in the reduction would break it.
    assert np.all(np.diff(C.detexp32(np.linspace(-20, 0, 100001, dtype=np.float32))) >= 0)


def test_dexp64_accuracy():
    x = np.linspace(-707.9, 0.0, 100001)
    y = C.dexp64(x)
    ref = np.array([math.exp(v) for v in x])
    assert np.max(np.abs(y - ref) / np.spacing(ref)) <= 2.0
    assert C.dexp64(np.array([0.0, -709.0, -np.inf, np.nan, 3.0])).tolist() == [1.0, 0.0, 0.0, 0.0, 1.0]


def test_quant40_dyadic_values():
    y = np.array([1.0, 0.5, 2.0**-40, 2.0**-41, 0.0, 0.75], dtype=np.float32)
    assert C.quant40(y).tolist() == [2**40, 2**39, 1, 0, 0, 3 * 2**38]
    assert C.quant40(np.array([1.0 - 2.0**-53])).tolist() == [2**40 - 1]


@pytest.mark.parametrize("weights", [[3, 0, 5, 2], [0, 0, 7], [1], [2**40, 1, 0, 2**39 + 5],
                                     [0, 1, 0, 0, 1, 0]])
def test_icdf_interval_closed_form(weights):
    """Token i is chosen exactly for r in [ceil(C_{i-1} 2^32 / Z), ceil(C_i 2^32 / Z))."""
    Z = sum(weights)
    cum = np.cumsum([0] + weights)
    for i, w in enumerate(weights):
        lo = -(-int(cum[i]) * 2**32 // Z)
        hi = -(-int(cum[i + 1]) * 2**32 // Z)
        if w == 0:
            assert lo == hi          # empty interval: zero-mass tokens are never drawn
            continue
        if lo == hi:                 # below the 32-bit resolution of r: only when w 2^32 < Z
            assert w * 2**32 < Z
            continue
        for r in {lo, hi - 1, (lo + hi) // 2}:
            assert C.icdf(weights, r) == i
    nz = [i for i, w in enumerate(weights) if w]
    assert C.icdf(weights, 0) == nz[0]
    assert C.icdf(weights, 2**32 - 1) == nz[-1]
    assert C.icdf([0, 0], 123) == -1


def test_accept_int_is_exact_u_less_than_p_over_q():
    rng = np.random.default_rng(3)
    for _ in range(3000):
        r = int(rng.integers(0, 2**32))
        q = int(rng.integers(0, 2**41))
        p = int(rng.integers(0, 2**41))
        if rng.random() < 0.1:
            p = q
        u = Fraction(r, 2**32)
        want = (p > 0) if q == 0 else (u < Fraction(p, q))
        assert C.accept_int(r, q, p) == want
    # Boundaries: u just below and at p/q.
    q, p = 3 * 2**30, 2**30          # p/q = 1/3
    r_edge = -(-(p * 2**32) // q)    # smallest r with r/2^32 >= 1/3
    assert C.accept_int(r_edge - 1, q, p) and not C.accept_int(r_edge, q, p)
    assert C.accept_int(2**32 - 1, q, q)      # p = q always accepts
    assert not C.accept_int(0, q, 0)          # p = 0 never accepts
