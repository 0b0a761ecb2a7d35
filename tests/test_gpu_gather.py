"""GPU parity of qgz_reduce_level_gather: P slices in separately allocated
buffers, read through device pointer tables, give the bits qgz_reduce_level
gives on the same slices back to back, and the oracle's."""
import numpy as np
import pytest
import torch

import oracle
import paper_2501_04266_amd as zq
from tests.gpu_util import assert_bits_equal, from_dev, poisoned, to_dev

pytestmark = pytest.mark.gpu


def _slices(P, m, block, seed):
    g = np.random.default_rng(seed)
    out = []
    for p in range(P):
        x = (g.standard_normal(m) * 10.0 ** g.uniform(-4, -1)).astype(np.float32)
        out.append(oracle.qgz_quantize(x, block))
    return out


# large (with and without leftover blocks), two-slice, small-level and ragged
# (generic kernel) launch shapes
CASES = [(1, 128, 4096), (2, 128, (1 << 23) + 4096), (8, 64, 1 << 20), (48, 128, 1179648), (5, 256, 3000),
         (8, 128, (1 << 23) + 4096), (3, 32, 65536 + 64)]


@pytest.mark.parametrize("P,block,m", CASES)
def test_gather_matches_contiguous_and_oracle(P, block, m):
    sl = _slices(P, m, block, 1000 + P + m)
    packed = [to_dev(a) for a, _ in sl]          # P separate allocations
    scales = [to_dev(b) for _, b in sl]
    gp, gs = zq.qgz_reduce_level_gather(packed, scales, m, block)
    cp, cs = zq.qgz_reduce_level(torch.cat(packed), torch.cat(scales), P, m, block)
    torch.cuda.synchronize()
    op, os_ = oracle.qgz_reduce_level(np.concatenate([a for a, _ in sl]), np.concatenate([b for _, b in sl]),
                                      P, m, block)
    assert_bits_equal(from_dev(gp), op, f"gather packed P={P} B={block} m={m}", block // 2)
    assert_bits_equal(from_dev(gs), os_, f"gather scales P={P} B={block} m={m}")
    assert from_dev(gp).tobytes() == from_dev(cp).tobytes() and from_dev(gs).tobytes() == from_dev(cs).tobytes()


def test_gather_from_views_and_graph_replay():
    """Slices as views at arbitrary (aligned) offsets of larger buffers, tables
    built once and reused from a captured HIP graph."""
    P, block, m = 4, 128, 1 << 18
    sl = _slices(P, m, block, 77)
    big = torch.zeros(P * (m // 2 + 4096), dtype=torch.uint8, device="cuda")
    bigs = torch.zeros(P * (m // block + 64), dtype=torch.float32, device="cuda")
    packed, scales = [], []
    for p, (a, b) in enumerate(sl):
        off, soff = p * (m // 2 + 4096) + 2048, p * (m // block + 64) + 16
        packed.append(big[off:off + m // 2])
        scales.append(bigs[soff:soff + m // block])
        packed[-1].copy_(to_dev(a))
        scales[-1].copy_(to_dev(b))
    tables = zq.gather_tables(packed, scales)
    op, os_ = oracle.qgz_reduce_level(np.concatenate([a for a, _ in sl]), np.concatenate([b for _, b in sl]),
                                      P, m, block)
    gp, gs = poisoned(m // 2, torch.uint8), poisoned(m // block, torch.float32)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            zq.qgz_reduce_level_gather(packed, scales, m, block, packed_out=gp, scales_out=gs, tables=tables)
    torch.cuda.synchronize()
    for rep in range(3):
        gp.zero_()
        gs.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert_bits_equal(from_dev(gp), op, f"replay {rep} packed", block // 2)
        assert_bits_equal(from_dev(gs), os_, f"replay {rep} scales")


def test_gather_binding_checks_and_raw_stream():
    """The binding rejects byte slices that are not 16-byte aligned where the
    vector path needs them (the library cannot read device-resident
    addresses), and a call on a raw stream handle keeps the tables it built
    alive until the kernel has run."""
    P, block, m = 3, 128, 1 << 16
    sl = _slices(P, m, block, 91)
    packed = [to_dev(a) for a, _ in sl]
    scales = [to_dev(b) for _, b in sl]
    big = torch.zeros(m // 2 + 16, dtype=torch.uint8, device="cuda")
    shifted = big[1:1 + m // 2]
    shifted.copy_(packed[1])
    with pytest.raises(ValueError):
        zq.qgz_reduce_level_gather([packed[0], shifted, packed[2]], scales, m, block)
    op, os_ = oracle.qgz_reduce_level(np.concatenate([a for a, _ in sl]), np.concatenate([b for _, b in sl]),
                                      P, m, block)
    gp, gs = poisoned(m // 2, torch.uint8), poisoned(m // block, torch.float32)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())      # the inputs' uploads and the poison fill
    for _ in range(3):
        zq.qgz_reduce_level_gather(packed, scales, m, block, packed_out=gp, scales_out=gs, stream=s.cuda_stream)
    s.synchronize()
    assert_bits_equal(from_dev(gp), op, "raw-stream gather packed", block // 2)
    assert_bits_equal(from_dev(gs), os_, "raw-stream gather scales")
