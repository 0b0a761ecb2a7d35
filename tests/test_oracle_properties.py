"""Property-based pins of the oracle against the brute-force definition
(tests/brute.py: exact rationals, its own decoding of the input bits):
random shapes for quantise, dequantise and the reduce level.  n runs from 0
to several blocks, with n = 0, n = 1, n < B, odd n and tails of 1 and B - 1
drawn deliberately; every power-of-two block from 32 to 1024; every input
kind of the brute-force cases (Gaussian, Student-t outliers, zero and -0
blocks, values around the 2^-119 flush threshold, exact .5 ties, constant
blocks) and every input / output type.  Hypothesis runs derandomised and
without its example database, so the CPU suite is reproducible."""
from hypothesis import given, settings
from hypothesis import strategies as st

from tests import pin_checks as pc

BLOCKS = [32, 64, 128, 256, 512, 1024]
KINDS = ["normal", "outlier", "zeros", "tiny", "ties", "const"]
SETTINGS = settings(max_examples=60, deadline=None, database=None, derandomize=True)


@st.composite
def shapes(draw, most=700):
    """(n, block) with the edge lengths drawn on purpose."""
    block = draw(st.sampled_from(BLOCKS))
    edge = st.builds(lambda k, t: k * block + t, st.integers(0, 2), st.sampled_from([0, 1, block - 1]))
    n = draw(st.one_of(st.integers(0, most), edge, st.sampled_from([0, 1, 2, 3])))
    return n, block


def _kind(n, kind):
    # the outlier and tie generators place a value at a fixed index
    return "normal" if n == 0 and kind in ("outlier", "ties") else kind


@SETTINGS
@given(op=st.sampled_from(["qwz", "qgz"]), dtype=st.sampled_from(["f32", "f16", "bf16"]), shape=shapes(),
       kind=st.sampled_from(KINDS), seed=st.integers(0, 2**31 - 1))
def test_quantize_matches_brute_force(op, dtype, shape, kind, seed):
    n, block = shape
    pc.check_brute_quantize(op, dtype, n, block, _kind(n, kind), seed)


@SETTINGS
@given(op=st.sampled_from(["qwz", "qgz"]), out=st.sampled_from(["f32", "f16", "bf16"]), shape=shapes(),
       kind=st.sampled_from(KINDS), seed=st.integers(0, 2**31 - 1))
def test_dequantize_matches_brute_force(op, out, shape, kind, seed):
    n, block = shape
    pc.check_brute_dequantize(op, n, block, _kind(n, kind), seed, out)


@settings(max_examples=40, deadline=None, database=None, derandomize=True)
@given(P=st.sampled_from([1, 2, 3, 4, 5, 8, 48]), shape=shapes(most=300), seed=st.integers(0, 2**31 - 1),
       identical=st.booleans())
def test_reduce_level_matches_brute_force(P, shape, seed, identical):
    m, block = shape
    if m == 0:
        m = 1
    pc.check_brute_reduce(P, m, block, seed, identical=identical)
