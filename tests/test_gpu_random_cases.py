"""Seeded random sweep over the calls' parameter space (sizes log-uniform
from 1 to ~3e5 elements, every block size, dtype and output type, P up to
64), each case bit for bit against the oracle.  Complements the hand-picked
edge cases with combinations nobody chose.  ZQ_RANDOM_CASES sets the count
(default 120), ZQ_RANDOM_SEED the seed of the case draws (default 2025)."""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2501_04266_amd as zq
from tests.gpu_util import assert_bits_equal, from_dev, to_dev

pytestmark = pytest.mark.gpu

BLOCKS = [32, 64, 128, 256, 512, 1024]
DT = ["f32", "f16", "bf16"]
TORCH = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def _x(g, n, dt):
    x = (g.standard_normal(n) * 10.0 ** g.uniform(-5, 1)).astype(np.float32)
    if n > 8 and g.random() < 0.3:
        x[g.integers(0, n, size=max(1, n // 1000))] *= 100.0       # outliers
    if n > 64 and g.random() < 0.3:
        s = int(g.integers(0, n - 32))
        x[s:s + 32] = 0.0                                         # a zero run
    if dt == "f16":
        return x.astype(np.float16)
    if dt == "bf16":
        return torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    return x


SEED = int(os.environ.get("ZQ_RANDOM_SEED", "2025"))


def _cases(count=int(os.environ.get("ZQ_RANDOM_CASES", "120")), seed=SEED):
    g = np.random.default_rng(seed)
    out = []
    for i in range(count):
        op = ["qwz", "qgz", "reduce", "fused", "gather"][i % 5]
        n = int(np.exp(g.uniform(0, np.log(300_000))))
        out.append((i, op, n, int(g.choice(BLOCKS)), str(g.choice(DT)), str(g.choice(DT)), int(g.integers(1, 65))))
    return out


@pytest.mark.parametrize("i,op,n,block,dt,out,P", _cases())
def test_random_case(i, op, n, block, dt, out, P):
    g = np.random.default_rng(10_000 + i if SEED == 2025 else [SEED, i])
    what = f"case {i}: {op} n={n} B={block} in={dt} out={out} P={P}"
    if op in ("qwz", "qgz"):
        x = _x(g, n, dt)
        xd = to_dev(x, dt)
        if op == "qwz":
            c, s = zq.qwz_quantize(xd, block)
            y = zq.qwz_dequantize(c, s, block, out_dtype=TORCH[out])
            oc, os_ = oracle.qwz_quantize(x, block, dt)
            oy = oracle.qwz_dequantize(oc, os_, block, out)
        else:
            c, s = zq.qgz_quantize(xd, block)
            y = zq.qgz_dequantize(c, s, n, block, out_dtype=TORCH[out])
            oc, os_ = oracle.qgz_quantize(x, block, dt)
            oy = oracle.qgz_dequantize(oc, os_, n, block, out)
        torch.cuda.synchronize()
        assert_bits_equal(from_dev(c), oc, what + " codes", block)
        assert_bits_equal(from_dev(s), os_, what + " scales")
        assert_bits_equal(from_dev(y), oy, what + " dequant")
        return
    m = max(1, n // P)
    q = [oracle.qgz_quantize(_x(g, m, "f32"), block) for _ in range(P)]
    pin, sin = np.concatenate([a for a, _ in q]), np.concatenate([b for _, b in q])
    op_, os_ = oracle.qgz_reduce_level(pin, sin, P, m, block)
    if op == "reduce":
        rp, rs = zq.qgz_reduce_level(to_dev(pin), to_dev(sin), P, m, block)
    elif op == "gather":
        rp, rs = zq.qgz_reduce_level_gather([to_dev(a) for a, _ in q], [to_dev(b) for _, b in q], m, block)
    else:
        y = zq.qgz_reduce_dequantize(to_dev(pin), to_dev(sin), P, m, block, out_dtype=TORCH[out])
        torch.cuda.synchronize()
        assert_bits_equal(from_dev(y), oracle.qgz_dequantize(op_, os_, m, block, out), what + " fused")
        return
    torch.cuda.synchronize()
    assert_bits_equal(from_dev(rp), op_, what + " packed", block // 2)
    assert_bits_equal(from_dev(rs), os_, what + " scales")
