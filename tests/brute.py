"""Exact-arithmetic brute-force model of the block quantiser, for tiny inputs.

Independent of oracle/zq_oracle.c: it shares no code with it and takes a
different route to every result.  Values are exact rationals (fractions);
each binary32 operation of the definition is modelled by computing the exact
result and rounding it once with `round_fmt` (a from-scratch
round-to-nearest-even onto a p-bit significand grid with subnormals).  Codes
are chosen by enumerating every code in [-qmax, qmax] and taking the nearest,
ties to the even code, rather than by calling a rounding function.

Definition modelled (block-wise symmetric quantisation, ZeRO++ as described
in the paper's Background section; per-block scales, Evaluations / Model
Convergence):
  a = max|x|; a < 2^-119 -> scale 0, codes 0; s = fl(a/qmax); r = fl(qmax/a);
  code = nearest integer in [-qmax, qmax] to fl(x * r);
  dequant y = cvt(fl(code * s));
  reduce level: acc = 0; for p ascending: acc = fl(acc + fl(q_p * s_p)); requant acc.
"""
from fractions import Fraction as Fr

import numpy as np

# (significand bits p, minimum normal exponent, maximum exponent)
FMT = {
    "f32": (24, -126, 127),
    "bf16": (8, -126, 127),
    "f16": (11, -14, 15),
}
INF = float("inf")
TINY = Fr(1, 2 ** 119)


def _floor_log2(a):
    """floor(log2(a)) for a positive Fraction, exactly."""
    e = a.numerator.bit_length() - a.denominator.bit_length()
    # now 2^(e-1) < a < 2^(e+1); fix up to 2^e <= a < 2^(e+1)
    if Fr(2) ** e > a:
        e -= 1
    return e


def round_fmt(x, fmt="f32"):
    """Nearest value of format `fmt` to the exact rational x, ties to even."""
    p, emin, emax = FMT[fmt]
    if x == 0:
        return Fr(0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = max(_floor_log2(a), emin)
    ulp = Fr(2) ** (e - (p - 1))
    k = a / ulp
    n = k.numerator // k.denominator
    rem = k - n
    if rem > Fr(1, 2) or (rem == Fr(1, 2) and n % 2 == 1):
        n += 1
    v = n * ulp
    if v >= Fr(2) ** (emax + 1):
        return sign * INF
    return sign * v


def fl(x):
    return round_fmt(x, "f32")


def exact_values(arr, dtype):
    """Exact rational value of each element of a numpy array."""
    if dtype == "bf16":
        f = (np.asarray(arr, np.uint16).astype(np.uint32) << 16).view(np.float32)
        return [Fr(float(v)) for v in f]
    return [Fr(float(v)) for v in np.asarray(arr)]


def nearest_code(t, qmax):
    return min(range(-qmax, qmax + 1), key=lambda c: (abs(t - c), c % 2))


def quantize_block(vals, qmax):
    a = max(abs(v) for v in vals)
    if a < TINY:
        return [0] * len(vals), Fr(0)
    s = fl(a / qmax)
    r = fl(Fr(qmax) / a)
    return [nearest_code(fl(v * r), qmax) for v in vals], s


def quantize(vals, block, qmax):
    codes, scales = [], []
    for b in range(0, len(vals), block):
        c, s = quantize_block(vals[b:b + block], qmax)
        codes += c
        scales.append(s)
    return codes, scales


def dequantize(codes, scales, block, out_fmt="f32"):
    """Exact dequantised values as Python floats.  A non-zero product that
    rounds to zero in the output format keeps its sign (-0.0), as IEEE
    rounding does; rationals alone cannot carry that sign."""
    out = []
    for i, q in enumerate(codes):
        prod = fl(Fr(q) * scales[i // block])
        v = round_fmt(prod, out_fmt)
        out.append(-0.0 if (v == 0 and prod < 0) else float(v))
    return out


def reduce_level(slices, block):
    """slices: list of (codes, scales) with equal lengths; returns requantised (codes, scales)."""
    m = len(slices[0][0])
    acc = []
    for i in range(m):
        s = Fr(0)
        for codes, scales in slices:
            s = fl(s + fl(Fr(codes[i]) * scales[i // block]))
        acc.append(s)
    return quantize(acc, block, 7)


def unpack_int4(packed, n):
    """Codes from packed bytes: element 2j = low nibble of byte j, two's complement."""
    out = []
    for k in range(n):
        byte = int(packed[k // 2])
        nib = (byte >> 4) if (k % 2) else (byte & 0xF)
        out.append(nib - 16 if nib >= 8 else nib)
    return out


def to_f32_bits(v):
    return int(np.float32(float(v)).view(np.uint32))


def to_out_bits(v, fmt):
    """Bit pattern of a value (Fraction or float, possibly -0.0) that is
    exactly representable in fmt."""
    if isinstance(v, float) and v == 0.0 and np.signbit(v):
        return {"f32": 0x80000000, "bf16": 0x8000, "f16": 0x8000}[fmt]
    if v in (INF, -INF):
        f = np.float32(v)
        return int(f.view(np.uint32)) >> 16 if fmt == "bf16" else (
            int(np.float16(v).view(np.uint16)) if fmt == "f16" else int(f.view(np.uint32)))
    v = Fr(v)
    if fmt == "f32":
        return to_f32_bits(v)
    if fmt == "bf16":
        u = to_f32_bits(v)
        assert u & 0xFFFF == 0, "value not representable in bf16"
        return u >> 16
    h = np.float16(float(v))
    assert Fr(float(h)) == v, "value not representable in f16"
    return int(h.view(np.uint16))
