"""Exhaustive CPU check of the kernels' block-scale shortcut.

The definition stores the block scale s = fl(a / qmax), a correctly rounded
binary32 division.  The HIP kernels compute it instead as one binary64
multiply by the binary64 constant fl64(1/qmax), rounded once to binary32
(three instructions instead of the division sequence).  The argument for
that is written beside the kernel; this test checks the claim itself for
every binary32 absmax the definition can meet: every finite a >= 2^-119
(smaller absmax values flush the block and never form a scale), for
qmax = 7 (INT4) and qmax = 127 (INT8).

Reference: fl32(fl64(a) / qmax).  A binary64 quotient rounded again to
binary32 is the correctly rounded binary32 quotient, because 53 >= 2*24 + 2
(innocuous double rounding for division, Figueroa 1995); a random sample is
also checked against exact rational arithmetic (tests/brute.py).
"""
from concurrent.futures import ThreadPoolExecutor
from fractions import Fraction as Fr

import numpy as np
import pytest

from tests import brute

LO = 0x04000000          # bit pattern of 2^-119
HI = 0x7F800000          # +inf (exclusive)
CHUNK = 1 << 24


def _mismatches(qmax, start):
    bits = np.arange(start, min(start + CHUNK, HI), dtype=np.uint32)
    a = bits.view(np.float32).astype(np.float64)
    shortcut = (a * (1.0 / qmax)).astype(np.float32)
    exact = (a / qmax).astype(np.float32)
    bad = np.flatnonzero(shortcut.view(np.uint32) != exact.view(np.uint32))
    return [int(bits[i]) for i in bad[:4]], int(bad.size)


def test_reference_is_correctly_rounded():
    g = np.random.default_rng(17)
    bits = g.integers(LO, HI, 4000, dtype=np.uint64).astype(np.uint32)
    for qmax in (7, 127):
        a = bits.view(np.float32)
        ref = (a.astype(np.float64) / qmax).astype(np.float32)
        for v, r in zip(a, ref):
            assert brute.to_f32_bits(brute.fl(Fr(float(v)) / qmax)) == int(r.view(np.uint32))


@pytest.mark.slow
@pytest.mark.parametrize("qmax", [7, 127])
def test_scale_shortcut_exhaustive(qmax):
    starts = range(LO, HI, CHUNK)
    with ThreadPoolExecutor(8) as ex:
        results = list(ex.map(lambda s: _mismatches(qmax, s), starts))
    total = sum(n for _, n in results)
    first = [b for bad, _ in results for b in bad][:4]
    assert total == 0, f"qmax={qmax}: {total} absmax values where the shortcut differs, e.g. {[hex(b) for b in first]}"
