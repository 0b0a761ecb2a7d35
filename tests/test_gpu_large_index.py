"""GPU parity beyond 2^31 elements: every kernel indexes elements, bytes and
blocks in 64 bits.  Each tensor has 2^31 + 4099 elements (a ragged last
block); outputs are compared bit for bit with the oracle over the whole
tensor.  Host memory peaks at about 20 GB per test."""
import numpy as np
import pytest
import torch

import oracle
import paper_2501_04266_amd as zq
from paper_2501_04266_amd import workloads as wl
from tests.gpu_util import assert_bits_equal, from_dev, to_dev

pytestmark = pytest.mark.gpu

N_BIG = (1 << 31) + 4099


def test_qwz_beyond_2g_elements():
    w = wl.weights(N_BIG, "bf16", key=[6, wl.ROLE_WEIGHT, 0, 0])
    codes, scales = zq.qwz_quantize(to_dev(w, "bf16"), 256)
    torch.cuda.synchronize()
    oc, os_ = oracle.qwz_quantize(w, 256, "bf16")
    del w
    assert_bits_equal(from_dev(codes), oc, "qwz codes, n > 2^31", 256)
    assert_bits_equal(from_dev(scales), os_, "qwz scales, n > 2^31")
    y = zq.qwz_dequantize(codes, scales, 256, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    del codes, scales
    assert_bits_equal(from_dev(y), oracle.qwz_dequantize(oc, os_, 256, "bf16"), "qwz dequant bf16, n > 2^31")


def test_qgz_beyond_2g_elements():
    g = wl.normal_f32(N_BIG, 1e-3, key=[6, wl.ROLE_OWN_GRAD, 0, 0])
    packed, scales = zq.qgz_quantize(to_dev(g), 128)
    torch.cuda.synchronize()
    op_, os_ = oracle.qgz_quantize(g, 128)
    del g
    assert_bits_equal(from_dev(packed), op_, "qgz packed, n > 2^31", 64)
    assert_bits_equal(from_dev(scales), os_, "qgz scales, n > 2^31")
    y = zq.qgz_dequantize(packed, scales, N_BIG, 128, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    del packed, scales
    assert_bits_equal(from_dev(y), oracle.qgz_dequantize(op_, os_, N_BIG, 128, "bf16"), "qgz dequant bf16, n > 2^31")


def test_reduce_level_beyond_2g_elements():
    """P = 2 random slices of m = 2^31 + 4096 elements (ragged: the last
    blocks fall outside whole tile groups), reduced and also fused with the
    final dequantisation to bf16."""
    P, m, block = 2, (1 << 31) + 4096, 128
    nb4, nsc = (m + 1) // 2, (m + block - 1) // block
    pin = wl.random_bytes(P * nb4, key=[6, wl.ROLE_MISC, 1, 0])
    sin = wl.uniform_f32(P * nsc, *wl.ALL_SHARES_SCALES, key=[6, wl.ROLE_MISC, 1, 1])
    dpin, dsin = torch.from_numpy(pin).cuda(), torch.from_numpy(sin).cuda()
    rp, rs = zq.qgz_reduce_level(dpin, dsin, P, m, block)
    y = zq.qgz_reduce_dequantize(dpin, dsin, P, m, block, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    del dpin, dsin
    orp, ors = oracle.qgz_reduce_level(pin, sin, P, m, block)
    del pin, sin
    assert_bits_equal(from_dev(rp), orp, "reduce packed, m > 2^31", 64)
    assert_bits_equal(from_dev(rs), ors, "reduce scales, m > 2^31")
    del rp, rs
    assert_bits_equal(from_dev(y), oracle.qgz_dequantize(orp, ors, m, block, "bf16"), "fused bf16, m > 2^31")
