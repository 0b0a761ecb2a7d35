"""CPU tests: the oracle against brute force, golden fixtures, closed forms,
invariants and library format conversions (see tests/pin_checks.py)."""
import numpy as np
import pytest

import oracle
from tests import pin_checks as pc


@pytest.mark.parametrize("case", pc.BRUTE_QUANT_CASES, ids=lambda c: "-".join(map(str, c)))
def test_brute_quantize(case):
    pc.check_brute_quantize(*case)


@pytest.mark.parametrize("case", pc.BRUTE_DEQ_CASES, ids=lambda c: "-".join(map(str, c)))
def test_brute_dequantize(case):
    pc.check_brute_dequantize(*case)


@pytest.mark.parametrize("case", pc.BRUTE_REDUCE_CASES, ids=lambda c: "-".join(map(str, c)))
def test_brute_reduce(case):
    pc.check_brute_reduce(*case)


@pytest.mark.parametrize("P", [2, 3, 8])
def test_brute_reduce_identical(P):
    pc.check_brute_reduce(P, 128, 64, 40 + P, identical=True)


def test_golden_fixtures():
    pc.check_golden()


def test_midpoints():
    pc.check_midpoints()


def test_closed_forms():
    pc.check_closed_forms()


def test_invariants():
    pc.check_invariants()


def test_reduce_invariants():
    pc.check_reduce_invariants()


def test_format_conversions():
    pc.check_format_conversions()


def test_size_ratios():
    pc.check_size_ratios()


def test_empty_and_errors():
    c, s = oracle.qwz_quantize(np.zeros(0, np.float32), 256)
    assert c.size == 0 and s.size == 0
    with pytest.raises(oracle.OracleError):
        oracle.qwz_quantize(np.zeros(4, np.float32), 3)


def test_threads_bit_identical():
    """OpenMP over blocks cannot change any bit: blocks are independent and the
    slice sum inside a block is sequential."""
    g = np.random.default_rng(3)
    x = (g.standard_normal(1 << 18) * 1e-3).astype(np.float32)
    t0 = oracle.get_threads()
    try:
        oracle.set_threads(1)
        a = oracle.qgz_quantize(x, 128)
        oracle.set_threads(max(2, t0))
        b = oracle.qgz_quantize(x, 128)
    finally:
        oracle.set_threads(t0)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1].view(np.uint32), b[1].view(np.uint32))
