"""The nucleus kernel's shortcut, checked on the CPU: every token whose bin
floor((m - s) * 2048 / 27.8) is at most 2000 has a positive integer mass
floor(detexp32(s - m) * 2^40), so once the cut's bin is one of those the later passes may test
the bin alone. Exhaustive over the binary32 values of d = s - m near the bin-2000 boundary, and
over every binary32 d in [-27.2, -20]; above -20 the mass exceeds 2^-40 by orders of magnitude.
"""
import numpy as np

from oracle import contract as C

BINS = 2048
SCALE = np.float32(BINS) / np.float32(27.8)   # the kernel's binary32 constant
SURE_BIN = 2000


def _bins(d):
    prod = (-d).astype(np.float32) * SCALE          # one binary32 product, as in the kernel
    return np.minimum(BINS - 1, np.trunc(prod).astype(np.int64))


def _floats_between(lo, hi):
    a = np.float32(lo).view(np.int32)
    b = np.float32(hi).view(np.int32)
    # negative floats: larger magnitude = larger bit pattern
    ints = np.arange(min(a, b), max(a, b) + 1, dtype=np.int64).astype(np.int32)
    return ints.view(np.float32)


def test_every_token_of_a_sure_bin_has_positive_mass():
    d = _floats_between(-27.2, -20.0)
    assert d.size > 3_000_000 and np.all(d < 0)
    b = _bins(d)
    sure = b <= SURE_BIN
    P = C.quant40(C.detexp32(d))
    assert np.all(P[sure] >= 1)
    # the boundary is inside the range: some d of bin 2001 exist, and bin 2000 is reached
    assert np.any(b == SURE_BIN) and np.any(b == SURE_BIN + 1)
    # the margin: the least d of a sure bin is above -27.17, where e^d > 1.5e-12 > 2^-40
    assert d[sure].min() > -27.17 and np.exp(np.float64(d[sure].min())) > 2.0 ** -40 * 1.5


def test_bins_are_non_increasing_in_d():
    d = np.sort(_floats_between(-27.8, -26.0))
    b = _bins(d)
    assert np.all(np.diff(b) <= 0)
