"""Checks that pin the CPU oracle to something other than itself.

Each check raises AssertionError on failure.  They are collected by
tests/test_oracle_pins.py and also run, in a child process, against
deliberately broken copies of the oracle (tests/test_oracle_mutants.py) to
show that a plausible mistake anywhere in the oracle is caught.

Pins used (none re-types the oracle's own formula):
  * brute force: tests/brute.py recomputes tiny cases in exact rational
    arithmetic with its own round-to-nearest-even and code enumeration;
  * hand-derived golden fixtures in tests/golden/ (worked by hand from the
    definition, derivation stored beside the values);
  * closed forms: all-zero block, single non-zero, constant block, absmax a
    power-of-two multiple of qmax;
  * invariants: absmax element -> +-qmax, |x - deq| <= s (1/2 + 2^-13),
    P identical slices keep their codes, x + (-x) gives a zero block;
  * library routines for the element formats: numpy float16 casts and torch
    bfloat16 casts (both round to nearest even).
"""
import json
import os
from fractions import Fraction as Fr

import numpy as np

import oracle
from tests import brute

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _bf16_bits(x32):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x32, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _as_dtype(x32, dtype):
    if dtype == "f32":
        return np.ascontiguousarray(x32, np.float32)
    if dtype == "f16":
        return x32.astype(np.float16)
    return _bf16_bits(x32)


def _tiny_inputs(seed, n, kind):
    g = _rng(seed)
    if kind == "normal":
        x = g.standard_normal(n).astype(np.float32) * np.float32(0.02)
    elif kind == "outlier":
        x = (g.standard_t(3, n) * 0.02).astype(np.float32)
        k = max(1, n // 50)
        x[g.choice(n, k, replace=False)] *= 100
    elif kind == "zeros":
        x = g.standard_normal(n).astype(np.float32)
        x[: min(n, 64)] = 0.0
        if n > 100:
            x[70:90] = -0.0
    elif kind == "tiny":
        # straddles the 2^-119 flush threshold and reaches fp32 subnormals
        e = g.integers(-150, -110, n)
        x = (g.choice([-1.0, 1.0], n) * np.ldexp(1.0 + g.random(n), e)).astype(np.float32)
    elif kind == "ties":
        # values landing exactly on .5 after scaling: absmax 7 or 127 and half-integers
        x = (g.integers(-14, 15, n) / 2.0).astype(np.float32)
        x[0] = 7.0
    elif kind == "const":
        x = np.full(n, np.float32(-0.37), np.float32)
    else:
        raise ValueError(kind)
    return x


# --------------------------------------------------------------------------
# brute-force pins
# --------------------------------------------------------------------------

def check_brute_quantize(op, dtype, n, block, kind, seed):
    x32 = _tiny_inputs(seed, n, kind)
    x = _as_dtype(x32, dtype)
    qmax = 127 if op == "qwz" else 7
    vals = brute.exact_values(x, dtype)
    bc, bs = brute.quantize(vals, block, qmax)
    if op == "qwz":
        codes, scales = oracle.qwz_quantize(x, block, dtype)
        oc = [int(c) for c in codes]
    else:
        packed, scales = oracle.qgz_quantize(x, block, dtype)
        oc = brute.unpack_int4(packed, n)
        if n % 2:
            assert int(packed[-1]) >> 4 == 0, "odd n: last high nibble must be 0"
    assert oc == bc, f"codes differ ({op} {dtype} n={n} B={block} {kind}): first at " \
                     f"{next(i for i in range(n) if oc[i] != bc[i])}"
    got = [int(v) for v in np.asarray(scales, np.float32).view(np.uint32)]
    want = [brute.to_f32_bits(s) for s in bs]
    assert got == want, f"scales differ ({op} {dtype} n={n} B={block} {kind})"
    return bc, bs


def check_brute_dequantize(op, n, block, kind, seed, out):
    x32 = _tiny_inputs(seed, n, kind)
    qmax = 127 if op == "qwz" else 7
    vals = brute.exact_values(x32, "f32")
    bc, bs = brute.quantize(vals, block, qmax)
    want = [brute.to_out_bits(v, out) for v in brute.dequantize(bc, bs, block, out)]
    if op == "qwz":
        codes, scales = oracle.qwz_quantize(x32, block, "f32")
        y = oracle.qwz_dequantize(codes, scales, block, out)
    else:
        packed, scales = oracle.qgz_quantize(x32, block, "f32")
        y = oracle.qgz_dequantize(packed, scales, n, block, out)
    got = [int(v) for v in (y.view(np.uint32) if out == "f32" else y.view(np.uint16))]
    assert got == want, f"dequant differs ({op} n={n} B={block} {kind} -> {out})"


def check_brute_reduce(P, m, block, seed, identical=False):
    g = _rng(seed)
    slices_x = [g.standard_normal(m).astype(np.float32) * np.float32(10.0 ** g.uniform(-4, 1)) for _ in range(P)]
    if identical:
        slices_x = [slices_x[0]] * P
    bq = []
    packs, scs = [], []
    for xs in slices_x:
        bq.append(brute.quantize(brute.exact_values(xs, "f32"), block, 7))
        p_, s_ = oracle.qgz_quantize(xs, block, "f32")
        packs.append(p_)
        scs.append(s_)
    bc, bs = brute.reduce_level(bq, block)
    op, os_ = oracle.qgz_reduce_level(np.concatenate(packs), np.concatenate(scs), P, m, block)
    oc = brute.unpack_int4(op, m)
    assert oc == bc, f"reduce codes differ (P={P} m={m} B={block})"
    assert [int(v) for v in os_.view(np.uint32)] == [brute.to_f32_bits(s) for s in bs], \
        f"reduce scales differ (P={P} m={m} B={block})"


def midpoint_block(qmax, block, seed):
    """A block whose elements sit within a few ulps of code midpoints
    (k + 1/2) * s, where multiplying by fl(qmax/a) and dividing by
    fl(a/qmax) can round to different codes.  Built in exact arithmetic
    (tests/brute.py); returns float32 values and the number of elements on
    which the two conventions disagree."""
    from fractions import Fraction as Fr
    g = _rng(seed)
    for _attempt in range(64):          # some absmax values never separate them
        a = Fr(float(np.float32(1.0 + g.random())))
        s = brute.fl(a / qmax)
        r = brute.fl(Fr(qmax) / a)
        vals, split = [a], 0
        while len(vals) < block:
            k = int(g.integers(0, qmax))
            mid = brute.fl((k + Fr(1, 2)) * s)
            x = mid + int(g.integers(-3, 4)) * Fr(2) ** (brute._floor_log2(mid) - 23)
            if x > a:
                continue
            x = x if g.random() < 0.5 else -x
            vals.append(x)
            split += brute.nearest_code(brute.fl(x * r), qmax) != brute.nearest_code(brute.fl(x / s), qmax)
        if split:
            break
    return np.array([float(v) for v in vals], np.float32), split


def check_midpoints():
    """Codes come from multiplying by the rounded reciprocal fl(qmax/a), not
    from dividing by the stored scale; the two differ near code midpoints."""
    for op, qmax, block, seed in (("qgz", 7, 128, 50), ("qwz", 127, 256, 51), ("qgz", 7, 64, 52)):
        x, split = midpoint_block(qmax, block, seed)
        assert split > 0, "midpoint block does not separate the two conventions"
        vals = brute.exact_values(x, "f32")
        bc, bs = brute.quantize(vals, block, qmax)
        if op == "qwz":
            codes, scales = oracle.qwz_quantize(x, block)
            oc = [int(c) for c in codes]
        else:
            packed, scales = oracle.qgz_quantize(x, block)
            oc = brute.unpack_int4(packed, x.size)
        assert oc == bc, f"midpoint codes differ ({op} B={block})"
        assert [int(v) for v in scales.view(np.uint32)] == [brute.to_f32_bits(v) for v in bs]


BRUTE_QUANT_CASES = [
    # (op, dtype, n, block, kind, seed)
    ("qgz", "f32", 1, 64, "normal", 1),
    ("qgz", "f32", 63, 64, "normal", 2),
    ("qgz", "f32", 129, 128, "outlier", 3),
    ("qgz", "f32", 300, 64, "zeros", 4),
    ("qgz", "f32", 257, 32, "tiny", 5),
    ("qgz", "f32", 128, 128, "ties", 6),
    ("qgz", "f16", 255, 128, "normal", 7),
    ("qgz", "bf16", 333, 64, "outlier", 8),
    ("qgz", "f32", 96, 32, "const", 9),
    ("qwz", "f32", 1, 256, "normal", 10),
    ("qwz", "f32", 513, 256, "outlier", 11),
    ("qwz", "f16", 300, 64, "normal", 12),
    ("qwz", "bf16", 700, 256, "zeros", 13),
    ("qwz", "f32", 260, 128, "tiny", 14),
    ("qwz", "f32", 256, 256, "ties", 15),
    ("qwz", "bf16", 64, 32, "const", 16),
]

BRUTE_DEQ_CASES = [
    ("qwz", 300, 256, "normal", 20, "f32"),
    ("qwz", 300, 64, "outlier", 21, "bf16"),
    ("qwz", 200, 128, "normal", 22, "f16"),
    ("qgz", 301, 64, "outlier", 23, "f32"),
    ("qgz", 256, 128, "normal", 24, "bf16"),
    ("qgz", 130, 32, "tiny", 25, "f16"),
]

BRUTE_REDUCE_CASES = [
    # (P, m, block, seed)
    (1, 200, 64, 30),
    (2, 257, 128, 31),
    (3, 96, 32, 32),
    (4, 128, 64, 33),
    (8, 300, 128, 34),
    (48, 64, 64, 35),
]


def check_golden():
    for fn in sorted(os.listdir(GOLDEN)):
        if not fn.endswith(".json"):
            continue
        d = json.load(open(os.path.join(GOLDEN, fn)))
        op = d.get("op")
        if op in ("qwz", "qgz"):
            B = d["block"]
            x = np.zeros(d["pad_zeros_to"], np.float32)
            x[: len(d["x"])] = d["x"]
            k = len(d["codes"])
            if op == "qwz":
                codes, sc = oracle.qwz_quantize(x, B)
                y = oracle.qwz_dequantize(codes, sc, B, "f32")
                got = [int(c) for c in codes[:k]]
            else:
                packed, sc = oracle.qgz_quantize(x, B)
                y = oracle.qgz_dequantize(packed, sc, x.size, B, "f32")
                got = brute.unpack_int4(packed, k)
                assert [int(b) for b in packed[: len(d["packed_head"])]] == d["packed_head"], fn
            assert got == d["codes"], fn
            assert [float(s) for s in sc] == d["scale"], fn
            assert [float(v) for v in y[: len(d["dequant_f32"])]] == d["dequant_f32"], fn
        elif op == "reduce":
            B, P, m = d["block"], d["P"], d["m"]
            codes = np.zeros((P, m), np.int64)
            for p, c in enumerate(d["slice_codes"]):
                codes[p, : len(c)] = c
            packed = np.zeros((P, (m + 1) // 2), np.uint8)
            for p in range(P):
                nib = codes[p] & 0xF
                packed[p] = (nib[0::2] | (nib[1::2] << 4)).astype(np.uint8)
            scales = np.array(d["slice_scales"], np.float32).reshape(P, 1)
            out, sc = oracle.qgz_reduce_level(packed, scales, P, m, B)
            k = len(d["codes"])
            assert brute.unpack_int4(out, k) == d["codes"], fn
            assert [float(s) for s in sc] == d["scale"], fn
            y = oracle.qgz_dequantize(out, sc, m, B, "f32")
            assert [float(v) for v in y[:k]] == d["dequant_f32"], fn
        else:
            bc = d["bf16_case"]
            y = oracle.qwz_dequantize(np.array(bc["codes"], np.int8), np.array([bc["scale"]], np.float32),
                                      bc["block"], "bf16")
            got = (y.astype(np.uint32) << 16).view(np.float32)
            assert [float(v) for v in got] == bc["bf16"], fn
            fc = d["f16_case"]
            nib = np.array(fc["codes"] + [0], np.int64) & 0xF
            packed = (nib[0::2] | (nib[1::2] << 4)).astype(np.uint8)
            y = oracle.qgz_dequantize(packed, np.array([fc["scale"]], np.float32), len(fc["codes"]), fc["block"], "f16")
            assert [int(v) for v in y.view(np.uint16)] == fc["f16_bits"], fn


# --------------------------------------------------------------------------
# closed forms
# --------------------------------------------------------------------------

def check_closed_forms():
    for op, qmax in (("qwz", 127), ("qgz", 7)):
        quant = oracle.qwz_quantize if op == "qwz" else oracle.qgz_quantize

        def codes_of(x, B):
            if op == "qwz":
                c, s = quant(x, B)
                return [int(v) for v in c], s
            p, s = quant(x, B)
            return brute.unpack_int4(p, x.size), s

        # all-zero (and negative-zero) block: scale 0, codes 0
        x = np.zeros(128, np.float32)
        x[5::7] = -0.0
        c, s = codes_of(x, 128)
        assert c == [0] * 128 and s[0] == 0 and not np.signbit(s[0])
        # a block below the 2^-119 flush threshold
        x = np.zeros(64, np.float32)
        x[3] = np.float32(2.0 ** -120)
        x[9] = -np.float32(2.0 ** -125)
        c, s = codes_of(x, 64)
        assert c == [0] * 64 and s[0] == 0
        # exactly at the threshold: not flushed, full-range code
        x[3] = np.float32(2.0 ** -119)
        c, s = codes_of(x, 64)
        assert c[3] == qmax and s[0] > 0
        # single non-zero value: +-qmax at its index, zeros elsewhere
        for v in (0.3, -1e-3, 3.0e5):
            x = np.zeros(256, np.float32)
            x[17] = v
            c, s = codes_of(x, 256)
            assert c[17] == (qmax if v > 0 else -qmax) and sum(map(abs, c)) == qmax
            assert s[0] == np.float32(np.float32(abs(v)) / np.float32(qmax))
        # constant block: every code sign(c) * qmax
        x = np.full(64, np.float32(-2.75), np.float32)
        c, _ = codes_of(x, 64)
        assert c == [-qmax] * 64
        # absmax = qmax * 2^k: r = 2^-k is exact, codes = rint(x 2^-k), dequant exact
        for k in (-20, -3, 0, 5):
            g = _rng(100 + k)
            x = (g.integers(-2 * qmax, 2 * qmax + 1, 64) * 2.0 ** (k - 1)).astype(np.float32)
            x[0] = qmax * 2.0 ** k
            c, s = codes_of(x, 64)
            assert s[0] == np.float32(2.0 ** k)
            t = x.astype(np.float64) * 2.0 ** -k
            assert c == [int(v) for v in np.rint(t)]      # numpy rint: half to even
            if op == "qwz":
                cc, ss = oracle.qwz_quantize(x, 64)
                y = oracle.qwz_dequantize(cc, ss, 64)
            else:
                pp, ss = oracle.qgz_quantize(x, 64)
                y = oracle.qgz_dequantize(pp, ss, 64, 64)
            assert np.array_equal(y.astype(np.float64), np.array(c) * 2.0 ** k)


# --------------------------------------------------------------------------
# invariants on larger random inputs
# --------------------------------------------------------------------------

def check_invariants(n=1 << 20, seed=7):
    g = _rng(seed)
    x = (g.standard_normal(n) * 0.02).astype(np.float32)
    x[g.choice(n, n // 1000, replace=False)] *= 100
    for op, qmax, B in (("qwz", 127, 256), ("qgz", 7, 128), ("qgz", 7, 64)):
        if op == "qwz":
            c, s = oracle.qwz_quantize(x, B)
            codes = c.astype(np.int64)
            y = oracle.qwz_dequantize(c, s, B)
        else:
            p, s = oracle.qgz_quantize(x, B)
            lo = (p & 0xF).astype(np.int64)
            hi = (p >> 4).astype(np.int64)
            codes = np.empty(2 * p.size, np.int64)
            codes[0::2], codes[1::2] = lo, hi
            codes = np.where(codes >= 8, codes - 16, codes)[:n]
            y = oracle.qgz_dequantize(p, s, n, B)
        xb = x.reshape(-1, B)
        cb = codes.reshape(-1, B)
        # the absmax element of every block maps to +-qmax
        am = np.argmax(np.abs(xb), axis=1)
        top = cb[np.arange(cb.shape[0]), am]
        assert np.array_equal(np.abs(top), np.full_like(top, qmax))
        assert np.array_equal(np.sign(top), np.sign(xb[np.arange(xb.shape[0]), am]).astype(np.int64))
        # |x - deq| <= s (1/2 + 2^-13) on binary32 dequant (derived bound)
        sb = np.repeat(s.astype(np.float64), B)
        err = np.abs(x.astype(np.float64) - y.astype(np.float64))
        assert np.all(err <= sb * (0.5 + 2.0 ** -13))
        # codes stay within +-qmax
        assert codes.min() >= -qmax and codes.max() <= qmax
    # rounding noise on Gaussian blocks is close to uniform on [-s/2, s/2]:
    # mean (err / s)^2 ~ 1/12 (a dropped or doubled scale factor breaks it)
    xg = (g.standard_normal(n) * 0.02).astype(np.float32)
    for op, B in (("qwz", 256), ("qgz", 128), ("qgz", 64)):
        if op == "qwz":
            c, s = oracle.qwz_quantize(xg, B)
            y = oracle.qwz_dequantize(c, s, B)
        else:
            p, s = oracle.qgz_quantize(xg, B)
            y = oracle.qgz_dequantize(p, s, n, B)
        sb = np.repeat(s.astype(np.float64), B)
        r2 = ((xg.astype(np.float64) - y.astype(np.float64)) / sb) ** 2
        assert abs(12.0 * np.mean(r2) - 1.0) < 0.05


def check_reduce_invariants(m=1 << 16, seed=9):
    g = _rng(seed)
    B = 128
    x = (g.standard_normal(m) * 1e-3).astype(np.float32)
    p0, s0 = oracle.qgz_quantize(x, B)
    d0 = oracle.qgz_dequantize(p0, s0, m, B)
    # P identical slices keep their codes; output scale ~ P * input scale
    for P in (1, 2, 3, 4, 8, 48):
        out, so = oracle.qgz_reduce_level(np.tile(p0, P), np.tile(s0, P), P, m, B)
        assert np.array_equal(out, p0), f"P={P}: identical slices changed codes"
        rel = np.abs(so.astype(np.float64) / (P * s0.astype(np.float64)) - 1.0)
        assert rel.max() < 16 * 2.0 ** -23
        if P <= 4:
            # with P <= 4 the sequential sum equals fl(P * deq) and the requantised
            # dequant reproduces it up to the scale's rounding
            y = oracle.qgz_dequantize(out, so, m, B)
            assert np.allclose(y, P * d0, rtol=4 * 2.0 ** -23, atol=0)
    # x + (-x): exact zero sum -> zero block (scale 0, codes 0)
    pn, sn = oracle.qgz_quantize(-x, B)
    out, so = oracle.qgz_reduce_level(np.concatenate([p0, pn]), np.concatenate([s0, sn]), 2, m, B)
    assert not out.any() and not so.any()
    # derived error bound: |deq(R) - sum_p x_p| <= sum_p s_p/2 + s_out/2 (+ a few ulps)
    xs = [(g.standard_normal(m) * 1e-3).astype(np.float32) for _ in range(8)]
    qs = [oracle.qgz_quantize(v, B) for v in xs]
    out, so = oracle.qgz_reduce_level(np.concatenate([q[0] for q in qs]), np.concatenate([q[1] for q in qs]), 8, m, B)
    y = oracle.qgz_dequantize(out, so, m, B).astype(np.float64)
    exact = np.sum([v.astype(np.float64) for v in xs], axis=0)
    bound = np.repeat(sum(q[1].astype(np.float64) for q in qs) / 2 + so.astype(np.float64) / 2, B)
    assert np.all(np.abs(y - exact) <= bound * (1 + 1e-5))


# --------------------------------------------------------------------------
# reduce-level edge inputs: sums below the flush threshold, huge scales
# --------------------------------------------------------------------------

def pack_int4(codes):
    """Two's-complement nibbles of an int array (last axis), element 2j in the
    low nibble of byte j; an odd length leaves the last high nibble 0."""
    c = np.asarray(codes, np.int64)
    if c.shape[-1] % 2:
        c = np.concatenate([c, np.zeros(c.shape[:-1] + (1,), np.int64)], axis=-1)
    nib = c & 0xF
    return (nib[..., 0::2] | (nib[..., 1::2] << 4)).astype(np.uint8)


def special_reduce_slices(kind, P, m, block, seed):
    """P INT4 slices of m elements (packed bytes [P * ceil(m/2)], scales
    [P * ceil(m/B)]) that drive a reduce level into its rare cases.

    'subthreshold': scales 2^-128 .. 2^-112 (some binary32 subnormals), one
      level per block shared by its slices, codes over the whole nibble range
      -8..7, and every odd slice cancelling most of the slice before it
      (negated codes, a scale within 1% of its scale; an unpaired last slice
      is 2^-12 smaller), so that many block sums are non-zero yet below the
      2^-119 flush threshold, others just above it, and some exactly zero.
    'huge': slice 0 with scales 2^122 .. 2^125 (binary32 overflows at
      2^128, so 16 times such a scale is not finite above 2^124) in the
      first half of the blocks and ordinary scales in the second half; the
      other slices have scales of 2^-30 .. 2^100, so every product and sum
      stays finite."""
    g = _rng(seed)
    nb = (m + block - 1) // block
    if kind == "subthreshold":
        codes = g.integers(-8, 8, (P, m))
        level = g.uniform(-127, -113, nb)               # shared by the slices of a block
        scales = np.exp2(level + g.uniform(-1, 1, (P, nb))).astype(np.float32)
        if P % 2:                                       # the unpaired last slice stays small
            scales[P - 1] = np.exp2(level - 12).astype(np.float32)
        for p in range(1, P, 2):
            keep = g.random(m) < 0.85
            codes[p] = np.where(keep, -np.clip(codes[p - 1], -7, 7), codes[p])
            near = (scales[p - 1].astype(np.float64) * (1 + g.uniform(-0.01, 0.01, nb))).astype(np.float32)
            same = g.random(nb) < 0.25
            scales[p] = np.where(same, scales[p - 1], near)
    elif kind == "huge":
        codes = g.integers(-7, 8, (P, m))
        scales = np.exp2(g.uniform(-30, 100, (P, nb))).astype(np.float32)
        big = np.exp2(g.uniform(122, 125, nb)).astype(np.float32)
        scales[0] = np.where(np.arange(nb) < nb // 2, big, scales[0])
    else:
        raise ValueError(kind)
    return pack_int4(codes).reshape(-1), scales.reshape(-1)


def reduce_sums_f32(packed, scales, P, m, block):
    """The level's binary32 sums, recomputed with numpy's float32 arithmetic
    (one rounding per multiply and per add, ascending slice order).  Used
    only to confirm that an edge-case input really reaches the case it is
    built for, never as an expected value."""
    pk = np.asarray(packed, np.uint8).reshape(P, -1)
    sc = np.asarray(scales, np.float32).reshape(P, -1)
    nib = np.empty((P, 2 * pk.shape[1]), np.int64)
    nib[:, 0::2], nib[:, 1::2] = pk & 0xF, pk >> 4
    q = np.where(nib >= 8, nib - 16, nib)[:, :m].astype(np.float32)
    s = np.repeat(sc, block, axis=1)[:, :m]
    acc = np.zeros(m, np.float32)
    with np.errstate(over="raise"):
        for p in range(P):
            acc = acc + q[p] * s[p]
    return acc


def subthreshold_block_counts(packed, scales, P, m, block):
    """(blocks whose sum is non-zero but below 2^-119, blocks at or above it)."""
    acc = np.abs(reduce_sums_f32(packed, scales, P, m, block).astype(np.float64))
    nb = (m + block - 1) // block
    pad = np.zeros(nb * block)
    pad[:m] = acc
    amax = pad.reshape(nb, block).max(axis=1)
    return int(np.count_nonzero((amax > 0) & (amax < 2.0 ** -119))), int(np.count_nonzero(amax >= 2.0 ** -119))


def check_brute_special_reduce():
    """The oracle's reduce level on sums below the flush threshold (incl.
    subnormal products) and on scales near the top of the binary32 range,
    against brute force."""
    for kind, P, m, block, seed in (("subthreshold", 2, 256, 32, 70), ("subthreshold", 3, 200, 64, 71),
                                    ("huge", 1, 96, 32, 72), ("huge", 2, 256, 64, 73)):
        pin, sin = special_reduce_slices(kind, P, m, block, seed)
        if kind == "subthreshold":
            low, high = subthreshold_block_counts(pin, sin, P, m, block)
            assert low > 0 and high > 0, "edge input misses the flush threshold"
        nb = (m + block - 1) // block
        pk = pin.reshape(P, -1)
        sl = [(brute.unpack_int4(pk[p], m), [Fr(float(v)) for v in sin[p * nb:(p + 1) * nb]]) for p in range(P)]
        bc, bs = brute.reduce_level(sl, block)
        op, os_ = oracle.qgz_reduce_level(pin, sin, P, m, block)
        assert brute.unpack_int4(op, m) == bc, f"reduce codes differ ({kind} P={P} m={m} B={block})"
        assert [int(v) for v in os_.view(np.uint32)] == [brute.to_f32_bits(s) for s in bs], \
            f"reduce scales differ ({kind} P={P} m={m} B={block})"


# --------------------------------------------------------------------------
# the multi-level chain
# --------------------------------------------------------------------------

CHAIN_CASES = [
    # (n, fan-ins, rank, block, seed)
    (2304, (3, 4, 3), 2, 32, 80),
    (3072, (2, 4, 3), 1, 64, 81),
]


def check_brute_chain(chain_fn=None, cases=CHAIN_CASES):
    """oracle.chain against a brute-force composition of the levels: the own
    gradient quantised, then per level the own chunk `rank` of the previous
    output (codes and scales cut at the same element offset) with seeded peer
    slices, reduced in exact arithmetic.  A non-zero rank exercises the chunk
    offsets."""
    chain_fn = chain_fn or oracle.chain
    for n, fanins, rank, block, seed in cases:
        g = _rng(seed)
        own = (g.standard_normal(n) * 1e-3).astype(np.float32)
        cur_c, cur_s = brute.quantize(brute.exact_values(own, "f32"), block, 7)
        op_, os_ = oracle.qgz_quantize(own, block)
        want, peers, cur_m = [], [], n
        for P in fanins:
            m = cur_m // P
            nbm = m // block
            slices, lvl = [], []
            for p in range(P):
                if p == rank:
                    slices.append((cur_c[rank * m:(rank + 1) * m], cur_s[rank * nbm:(rank + 1) * nbm]))
                    lvl.append(None)
                else:
                    x = (g.standard_normal(m) * 10.0 ** g.uniform(-4, 0)).astype(np.float32)
                    slices.append(brute.quantize(brute.exact_values(x, "f32"), block, 7))
                    lvl.append(oracle.qgz_quantize(x, block))
            cur_c, cur_s = brute.reduce_level(slices, block)
            want.append((m, cur_c, cur_s))
            peers.append(lvl)
            cur_m = m
        outs = chain_fn(op_, os_, n, list(fanins), peers, rank, block)
        assert len(outs) == len(fanins), "chain: wrong number of levels"
        for k, ((m, bc, bs), (gp, gs, gm)) in enumerate(zip(want, outs)):
            assert gm == m, f"chain level {k}: size {gm}, want {m}"
            assert brute.unpack_int4(gp, m) == bc, f"chain level {k} codes differ (rank {rank})"
            assert [int(v) for v in np.asarray(gs, np.float32).view(np.uint32)] == [brute.to_f32_bits(s) for s in bs], \
                f"chain level {k} scales differ (rank {rank})"


# --------------------------------------------------------------------------
# element formats against library conversions
# --------------------------------------------------------------------------

def _format_probe_values(seed=11, n=40000):
    g = _rng(seed)
    bits = g.integers(0, 2 ** 32, n, dtype=np.uint64).astype(np.uint32)
    v = bits.view(np.float32)
    v = v[np.isfinite(v)]
    special = np.array([0.0, -0.0, 1.0, 65504.0, 65519.99, 65520.0, 65536.0, 2.0 ** -24, 2.0 ** -25,
                        3 * 2.0 ** -25, 2.0 ** -14, 2.0 ** -14 - 2.0 ** -25, 6.0e-8, 1.00390625,
                        1.001953125, 3.01171875, 127.49609375, 3.0e38, -1.5e-40], np.float32)
    small = (g.standard_normal(20000) * 10.0 ** g.uniform(-9, 5, 20000)).astype(np.float32)
    return np.concatenate([v, special, -special, small]).astype(np.float32)


def check_format_conversions():
    import torch
    v = _format_probe_values()
    # f32 -> f16 against numpy's cast (round to nearest even)
    got = np.array([oracle.f32_to_f16_bits(float(a)) for a in v], np.uint16)
    with np.errstate(over="ignore"):
        want = v.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, want), "f32->f16 differs from numpy"
    # f32 -> bf16 against torch's cast (round to nearest even)
    got = np.array([oracle.f32_to_bf16_bits(float(a)) for a in v], np.uint16)
    want = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, want), "f32->bf16 differs from torch"
    # f16 -> f32, all finite patterns, against numpy's widening
    h = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    hf = h.view(np.float16)
    fin = np.isfinite(hf)
    got = np.array([oracle.f16_bits_to_f32(int(b)) for b in h[fin]], np.float32)
    assert np.array_equal(got.view(np.uint32), hf[fin].astype(np.float32).view(np.uint32))


def check_size_ratios():
    """Wire sizes against the volume reductions the paper states: INT8 halves
    the FP16 Allgather volume (Background; Communication Volume Analysis), INT4
    quarters the gradient volume.  Scales add 4/B bytes per element."""
    n = 452_984_832
    int8_bytes = n + 4 * oracle.num_scales(n, 256)
    int4_bytes = oracle.int4_bytes(n) + 4 * oracle.num_scales(n, 128)
    assert abs(int8_bytes / (2 * n) - (0.5 + 2 / 256)) < 1e-9
    assert abs(int4_bytes / (2 * n) - (0.25 + 2 / 128)) < 1e-9
    x = np.zeros(1000, np.float32)
    c, s = oracle.qwz_quantize(x, 256)
    assert c.nbytes == 1000 and s.size == 4
    p, s = oracle.qgz_quantize(x[:999], 64)
    assert p.nbytes == 500 and s.size == 16


ALL = [
    ("golden", check_golden),
    ("midpoints", check_midpoints),
    ("closed_forms", check_closed_forms),
    ("brute_quant", lambda: [check_brute_quantize(*c) for c in BRUTE_QUANT_CASES]),
    ("brute_dequant", lambda: [check_brute_dequantize(*c) for c in BRUTE_DEQ_CASES]),
    ("brute_reduce", lambda: [check_brute_reduce(*c) for c in BRUTE_REDUCE_CASES]),
    ("invariants", lambda: check_invariants(n=1 << 18)),
    ("reduce_invariants", lambda: check_reduce_invariants(m=1 << 14)),
    ("brute_special_reduce", check_brute_special_reduce),
    ("brute_chain", check_brute_chain),
    ("formats", check_format_conversions),
]


def run_all(stop_at_first=False):
    """Run every check; return the names of those that failed."""
    failed = []
    for name, fn in ALL:
        try:
            fn()
        except AssertionError:
            failed.append(name)
        except Exception as e:  # a crash also counts as detection
            failed.append(f"{name}:{type(e).__name__}")
        if failed and stop_at_first:
            break
    return failed


if __name__ == "__main__":
    import sys
    print(json.dumps(run_all(stop_at_first="--first" in sys.argv)))
