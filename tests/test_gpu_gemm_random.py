"""Seeded random sweep of the dequantise-on-load GEMM (qwz_dequant_gemm) over
its paths -- the weight-streaming kernel (M <= 16), the ping-pong kernel's
128 x 256 (17-128 rows) and 256 x 256 tiles, with and without K split across
workgroups -- with ragged M and N, K up to
3072, every block size and both input types.  Exact inputs (x = a/4 with
|a| <= 16, scales 2^-7, so every dequantised weight q/128 and every partial
sum, a multiple of 2^-9 below 2^15, is exact in binary32) make each case
bit for bit comparable with the oracle whatever order the matrix cores add
in.  Complements the hand-picked shapes with tile-edge, split and
workgroup-mapping remainders nobody chose.  ZQ_GEMM_RANDOM_CASES sets the
count (default 40)."""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2501_04266_amd as zq
from paper_2501_04266_amd import workloads as wl
from tests.gpu_util import from_dev, to_dev

pytestmark = pytest.mark.gpu

BLOCKS = [32, 64, 128, 256, 512, 1024]


def _cases(count=int(os.environ.get("ZQ_GEMM_RANDOM_CASES", "40")), seed=4266):
    g = np.random.default_rng(seed)
    out = []
    for i in range(count):
        band = i % 3
        M = int(g.integers(1, 65)) if band == 0 else int(g.integers(65, 513)) if band == 1 else int(g.integers(513, 1601))
        N = int(g.integers(1, 701))
        K = 64 * int(g.integers(1, 49))
        B = int(g.choice(BLOCKS))
        dt = str(g.choice(["bf16", "f16"]))
        out.append((i, M, N, K, B, dt))
    return out


@pytest.mark.parametrize("case", _cases(), ids=lambda c: "i{}-M{}-N{}-K{}-B{}-{}".format(*c))
def test_random_gemm_case(case):
    i, M, N, K, B, dt = case
    g = np.random.default_rng(10_000 + i)
    x = wl.to_storage((g.integers(-16, 17, M * K) / 4.0).astype(np.float32), dt).reshape(M, K)
    codes = g.integers(-127, 128, N * K).astype(np.int8)
    scales = np.full(-(-(N * K) // B), 2.0 ** -7, np.float32)
    want = oracle.qwz_dequant_gemm(x, codes, scales, N, B, dt)
    y = zq.qwz_dequant_gemm(to_dev(x, dt).reshape(M, K), to_dev(codes), to_dev(scales), N, B)
    torch.cuda.synchronize()
    got = from_dev(y).astype(np.float64)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"case {case}: {bad.size} of {got.size} differ; first at {np.unravel_index(bad[0], got.shape)}"
