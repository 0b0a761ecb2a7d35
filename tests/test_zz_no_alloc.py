"""GPU parity of the allocation-free gathered reduce
(qgz_reduce_level_gather_noalloc), called through the C ABI with host
arrays of slice addresses, against the existing gathered reduce
(qgz_reduce_level_gather, device tables) and the oracle.  Several calls in
a row, each smaller than the one before, so a call that read a stale entry
of the shared device table left by a larger earlier call would fail."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2501_04266_amd as zq
from paper_2501_04266_amd import _lib
from tests.gpu_util import assert_bits_equal, from_dev, poisoned, to_dev

pytestmark = pytest.mark.gpu


def _slices(P, m, block, seed):
    g = np.random.default_rng(seed)
    out = []
    for _ in range(P):
        x = (g.standard_normal(m) * 10.0 ** g.uniform(-4, -1)).astype(np.float32)
        out.append(oracle.qgz_quantize(x, block))
    return out


def _noalloc(packed, scales, m, block, po, so):
    P = len(packed)
    tab = (ctypes.c_void_p * P)(*[t.data_ptr() for t in packed])
    stab = (ctypes.c_void_p * P)(*[t.data_ptr() for t in scales])
    st = _lib.lib().qgz_reduce_level_gather_noalloc(ctypes.cast(tab, ctypes.c_void_p), ctypes.cast(stab, ctypes.c_void_p),
                                                    P, m, block, po.data_ptr(), so.data_ptr(),
                                                    torch.cuda.current_stream().cuda_stream)
    assert st == 0, _lib.lib().zq_status_string(st)


# (P, m, block) in order of decreasing input size: the largest P the table
# holds; a large level on the vector path; a ragged level (generic kernel)
CALLS = [(1024, 16384, 128), (8, (1 << 20) + 4096, 128), (3, 65536 + 77, 64)]


def test_noalloc_matches_gather_calls_in_a_row():
    for i, (P, m, block) in enumerate(CALLS):
        what = f"call {i}: P={P} m={m} B={block}"
        print(what, flush=True)
        sl = _slices(P, m, block, 500 + i)
        packed = [to_dev(a) for a, _ in sl]
        scales = [to_dev(b) for _, b in sl]
        gp, gs = zq.qgz_reduce_level_gather(packed, scales, m, block)
        po, so = poisoned(zq.int4_bytes(m), torch.uint8), poisoned(zq.num_scales(m, block), torch.float32)
        _noalloc(packed, scales, m, block, po, so)
        torch.cuda.synchronize()
        assert_bits_equal(from_dev(po), from_dev(gp), f"{what} packed vs gather", block // 2)
        assert_bits_equal(from_dev(so), from_dev(gs), f"{what} scales vs gather")
        op, os_ = oracle.qgz_reduce_level(np.concatenate([a for a, _ in sl]), np.concatenate([b for _, b in sl]),
                                          P, m, block)
        assert_bits_equal(from_dev(po), op, f"{what} packed vs oracle", block // 2)
        assert_bits_equal(from_dev(so), os_, f"{what} scales vs oracle")


def test_noalloc_binding_and_errors():
    """The Python binding passes caller outputs only; argument errors come
    back as ZQError before anything is enqueued."""
    P, m, block = 4, 1 << 16, 128
    sl = _slices(P, m, block, 77)
    packed = [to_dev(a) for a, _ in sl]
    scales = [to_dev(b) for _, b in sl]
    po, so = poisoned(m // 2, torch.uint8), poisoned(m // block, torch.float32)
    zq.qgz_reduce_level_gather_noalloc(packed, scales, m, block, po, so)
    torch.cuda.synchronize()
    op, os_ = oracle.qgz_reduce_level(np.concatenate([a for a, _ in sl]), np.concatenate([b for _, b in sl]),
                                      P, m, block)
    assert_bits_equal(from_dev(po), op, "binding packed", block // 2)
    assert_bits_equal(from_dev(so), os_, "binding scales")
    with pytest.raises(zq.ZQError):
        zq.qgz_reduce_level_gather_noalloc(packed, scales, m, block, packed[0], so)   # output over an input
