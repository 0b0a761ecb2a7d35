"""Pins of the oracle's dequantise-on-load GEMM (y = x @ deq(W)^T) against
facts that do not come from its own code: a brute-force rational sum, a
permutation weight, and block scales that span rows."""
import struct
from fractions import Fraction

import numpy as np

import oracle


def _bf16_bits(vals):
    """float values that are exact in bfloat16 -> uint16 bit patterns"""
    out = []
    for v in vals:
        (u,) = struct.unpack("<I", struct.pack("<f", float(v)))
        assert u & 0xFFFF == 0, v
        out.append(u >> 16)
    return np.array(out, np.uint16)


def _bf16_value(bits):
    return struct.unpack("<f", struct.pack("<I", int(bits) << 16))[0]


def test_brute_force_rational():
    rng = np.random.default_rng(5)
    M, N, K, B = 3, 5, 64, 32
    x = _bf16_bits(rng.integers(-40, 41, M * K) / 8.0).reshape(M, K)
    codes = rng.integers(-127, 128, N * K).astype(np.int8)
    scales = (rng.uniform(1e-3, 1e-1, (N * K) // B)).astype(np.float32)
    y = oracle.qwz_dequant_gemm(x, codes, scales, N, B, "bf16")
    wbits = oracle.qwz_dequantize(codes, scales, B, "bf16")
    for m in range(M):
        for n in range(N):
            exact = sum(Fraction(_bf16_value(x[m, k])) * Fraction(_bf16_value(wbits[n * K + k])) for k in range(K))
            bound = sum(abs(Fraction(_bf16_value(x[m, k])) * Fraction(_bf16_value(wbits[n * K + k])))
                        for k in range(K))
            assert abs(Fraction(y[m, n]) - exact) <= bound * Fraction(K, 2 ** 52)


def test_permutation_weight_selects_columns():
    rng = np.random.default_rng(6)
    M, N, K = 4, 64, 64
    perm = rng.permutation(K)[:N]
    codes = np.zeros(N * K, np.int8)
    codes[np.arange(N) * K + perm] = 1
    scales = np.ones((N * K) // 64, np.float32)        # w = q exactly
    x = _bf16_bits(rng.integers(-100, 101, M * K) / 4.0).reshape(M, K)
    y = oracle.qwz_dequant_gemm(x, codes, scales, N, 64, "bf16")
    xf = np.array([[_bf16_value(b) for b in row] for row in x])
    assert np.array_equal(y, xf[:, perm])


def test_block_scales_spanning_rows():
    # K = 64 and B = 128: block b covers rows 2b and 2b + 1
    M, N, K, B = 2, 6, 64, 128
    codes = np.ones(N * K, np.int8)
    scales = np.array([2.0 ** -j for j in range((N * K) // B)], np.float32)
    x = np.full((M, K), 0x3F80, np.uint16)            # bf16 1.0
    y = oracle.qwz_dequant_gemm(x, codes, scales, N, B, "bf16")
    for n in range(N):
        assert np.all(y[:, n] == K * 2.0 ** -(n // 2))


def test_fp16_inputs():
    rng = np.random.default_rng(7)
    M, N, K, B = 2, 3, 64, 64
    x = (rng.integers(-8, 9, (M, K)) / 4.0).astype(np.float16)
    codes = rng.integers(-127, 128, N * K).astype(np.int8)
    scales = np.full((N * K) // B, 2.0 ** -7, np.float32)   # w = q / 128, exact in fp16
    y = oracle.qwz_dequant_gemm(x, codes, scales, N, B, "f16")
    want = x.astype(np.float64) @ (codes.reshape(N, K).astype(np.float64) / 128.0).T
    assert np.array_equal(y, want)
