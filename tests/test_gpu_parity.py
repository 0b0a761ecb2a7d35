"""GPU parity: every HIP entry point, called through the C ABI, against the
CPU oracle on the same seeded host inputs.  Bit-exact on codes, packed bytes,
scales and dequantised outputs (fp32 / bf16 / fp16 bit patterns).

Sizes span several wave tiles and ragged tails (n not a multiple of the
block, odd n for INT4, slices that are not 16-byte aligned), every block
size, every element dtype, and the degenerate inputs of the method (zero and
sub-threshold blocks, exact ties, elements at code midpoints, outliers).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2501_04266_amd as zq
from tests import pin_checks as pc
from tests.gpu_util import assert_bits_equal, from_dev, poisoned, to_dev

pytestmark = pytest.mark.gpu

KINDS = ["normal", "outlier", "zeros", "tiny", "ties", "const"]


def _input(n, kind, seed, dtype):
    x32 = pc._tiny_inputs(seed, n, kind) if n else np.zeros(0, np.float32)
    return pc._as_dtype(x32, dtype)


def _run_quant(op, x_np, dtype, block):
    x = to_dev(x_np, dtype)
    if op == "qwz":
        c, s = zq.qwz_quantize(x, block)
    else:
        c, s = zq.qgz_quantize(x, block)
    torch.cuda.synchronize()
    return from_dev(c), from_dev(s)


def _oracle_quant(op, x_np, dtype, block):
    return (oracle.qwz_quantize if op == "qwz" else oracle.qgz_quantize)(x_np, block, dtype)


QUANT_CASES = []
for op in ("qwz", "qgz"):
    for dtype in ("f32", "bf16", "f16"):
        for block in (32, 64, 128, 256, 512, 1024):
            for n in (1, 17, 1024 * 3 + 5, 65536 + 1021):
                QUANT_CASES.append((op, dtype, block, n))


@pytest.mark.parametrize("op,dtype,block,n", QUANT_CASES)
def test_quantize_parity(op, dtype, block, n):
    for i, kind in enumerate(KINDS):
        x = _input(n, kind, 1000 * block + n + i, dtype)
        gc, gs = _run_quant(op, x, dtype, block)
        oc, os_ = _oracle_quant(op, x, dtype, block)
        assert_bits_equal(gc, oc, f"{op} codes {dtype} B={block} n={n} {kind}", block if op == "qwz" else block // 2)
        assert_bits_equal(gs, os_, f"{op} scales {dtype} B={block} n={n} {kind}")


@pytest.mark.parametrize("op,block", [("qwz", 256), ("qgz", 128), ("qgz", 64), ("qwz", 32)])
def test_quantize_midpoints(op, block):
    qmax = 127 if op == "qwz" else 7
    xs = [pc.midpoint_block(qmax, block, 60 + k)[0] for k in range(6)]
    x = np.concatenate(xs)
    gc, gs = _run_quant(op, x, "f32", block)
    oc, os_ = _oracle_quant(op, x, "f32", block)
    assert_bits_equal(gc, oc, f"{op} midpoint codes")
    assert_bits_equal(gs, os_, f"{op} midpoint scales")


def test_quantize_large_ragged():
    g = np.random.default_rng(5)
    n = (1 << 22) + 777
    x = (g.standard_normal(n) * 0.02).astype(np.float32)
    x[g.choice(n, n // 1000, replace=False)] *= 100
    for op, block in (("qwz", 256), ("qgz", 128), ("qgz", 64)):
        gc, gs = _run_quant(op, x, "f32", block)
        oc, os_ = _oracle_quant(op, x, "f32", block)
        assert_bits_equal(gc, oc, f"{op} codes large")
        assert_bits_equal(gs, os_, f"{op} scales large")


DEQ_CASES = []
for op in ("qwz", "qgz"):
    for out in ("f32", "bf16", "f16"):
        for block in (32, 128, 256, 1024):
            for n in (1, 15, 16, 33, 4096 * 3 + 7, 65536 + 1021):
                DEQ_CASES.append((op, out, block, n))


@pytest.mark.parametrize("op,out,block,n", DEQ_CASES)
def test_dequantize_parity(op, out, block, n):
    for i, kind in enumerate(("normal", "outlier", "tiny", "zeros")):
        x = _input(n, kind, 7000 + n + block + i, "f32")
        if op == "qwz":
            c, s = oracle.qwz_quantize(x, block)
            want = oracle.qwz_dequantize(c, s, block, out)
            y = zq.qwz_dequantize(to_dev(c), to_dev(s), block, out_dtype={"f32": torch.float32, "bf16": torch.bfloat16,
                                                                           "f16": torch.float16}[out])
        else:
            c, s = oracle.qgz_quantize(x, block)
            want = oracle.qgz_dequantize(c, s, n, block, out)
            y = zq.qgz_dequantize(to_dev(c), to_dev(s), n, block, out_dtype={"f32": torch.float32,
                                                                              "bf16": torch.bfloat16,
                                                                              "f16": torch.float16}[out])
        torch.cuda.synchronize()
        assert_bits_equal(from_dev(y), want, f"{op} dequant -> {out} B={block} n={n} {kind}")


def test_dequantize_golden_rounding():
    """Output narrowing ties (bf16 and f16 subnormal) on the GPU."""
    c = np.array([1, 3, -1, 127] + [0] * 252, np.int8)
    s = np.array([1.00390625], np.float32)
    y = zq.qwz_dequantize(to_dev(c), to_dev(s), 256, out_dtype=torch.bfloat16)
    assert_bits_equal(from_dev(y), oracle.qwz_dequantize(c, s, 256, "bf16"), "bf16 ties")
    nib = np.array([1, 3, -1, 0] + [0] * 28, np.int64) & 0xF
    packed = (nib[0::2] | (nib[1::2] << 4)).astype(np.uint8)
    s = np.array([2.0 ** -25], np.float32)
    y = zq.qgz_dequantize(to_dev(packed), to_dev(s), 32, 32, out_dtype=torch.float16)
    assert_bits_equal(from_dev(y), oracle.qgz_dequantize(packed, s, 32, 32, "f16"), "f16 subnormal ties")


def _f16_tie_cases(qmax, count, seed):
    """(code, scale) pairs whose binary32 product is an exact binary16 tie
    (13 dropped bits = 1000000000000b) in the normal range and is itself a
    rounded value, so rounding the exact product once to binary16 can give a
    different answer than the definition (round to binary32, then to
    binary16).  Found by search on the CPU."""
    g = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        q = g.integers(1, qmax + 1, 1 << 20) * g.choice([-1, 1], 1 << 20)
        s = (2.0 ** g.uniform(-10, -4, 1 << 20)).astype(np.float32)
        prod = (q.astype(np.float32) * s).astype(np.float32)
        u = prod.view(np.uint32)
        exact = q.astype(np.float64) * s.astype(np.float64)
        hit = ((u & 0x1FFF) == 0x1000) & (np.abs(prod) >= 2.0 ** -14) & (exact != prod.astype(np.float64))
        for i in np.flatnonzero(hit):
            out.append((int(q[i]), float(s[i])))
    return out[:count]


@pytest.mark.parametrize("op", ["qwz", "qgz"])
def test_dequantize_f16_ties_of_fp32_products(op):
    """Regression: fp16 output must round the binary32 product, not the exact
    one (a fused multiply-narrow instruction gets these wrong)."""
    block, nblk = 32, 256
    cases = _f16_tie_cases(127 if op == "qwz" else 7, nblk, 77)
    g = np.random.default_rng(3)
    codes = g.integers(-7, 8, nblk * block).astype(np.int64)
    scales = np.array([s for _, s in cases], np.float32)
    codes[::block] = [q for q, _ in cases]
    if op == "qwz":
        c = codes.astype(np.int8)
        want = oracle.qwz_dequantize(c, scales, block, "f16")
        y = zq.qwz_dequantize(to_dev(c), to_dev(scales), block, out_dtype=torch.float16)
    else:
        nib = codes & 0xF
        c = (nib[0::2] | (nib[1::2] << 4)).astype(np.uint8)
        want = oracle.qgz_dequantize(c, scales, codes.size, block, "f16")
        y = zq.qgz_dequantize(to_dev(c), to_dev(scales), codes.size, block, out_dtype=torch.float16)
    torch.cuda.synchronize()
    assert_bits_equal(from_dev(y), want, f"{op} f16 ties")


def _slices(P, m, block, seed, scale_spread=True):
    g = np.random.default_rng(seed)
    xs = []
    for p in range(P):
        sd = 10.0 ** g.uniform(-4, 0) if scale_spread else 1e-3
        x = (g.standard_normal(m) * sd).astype(np.float32)
        if m > 4 * block:
            x[block:2 * block] = 0.0          # a zero block in every slice
        xs.append(x)
    q = [oracle.qgz_quantize(x, block) for x in xs]
    return np.concatenate([a for a, _ in q]), np.concatenate([b for _, b in q])


REDUCE_CASES = []
for P in (1, 2, 3, 4, 8, 48):
    for block in (32, 64, 128, 256, 1024):
        for m in (32, 2048 * 3 + block, 65536 + 128):
            REDUCE_CASES.append((P, block, m))
# levels large enough for the 32-elements-per-lane variant (>= 4096 waves)
for P, block, m in ((3, 128, (1 << 23) + 4096), (2, 64, (1 << 23) + 2048), (2, 256, (1 << 24) + 256),
                    (1, 128, (1 << 23) + 4096), (2, 32, (1 << 22) + 1024)):
    REDUCE_CASES.append((P, block, m))
# batches that do not divide P (odd job counts in the pipelined kernel), and
# the largest P the ABI accepts, on the small-level and the generic path
for P, block, m in ((5, 128, (1 << 23) + 4096), (9, 64, 1 << 23), (17, 128, 4096 * 8),
                    (1024, 128, 8192), (1024, 64, 1000)):
    REDUCE_CASES.append((P, block, m))
# ragged m: not a multiple of the block, of 32, odd
for P, block, m in ((2, 128, 1000), (3, 64, 999), (8, 128, 65536 + 77), (48, 64, 4095), (5, 1024, 3000),
                    (4, 32, 33), (2, 256, 1)):
    REDUCE_CASES.append((P, block, m))


@pytest.mark.parametrize("P,block,m", REDUCE_CASES)
def test_reduce_level_parity(P, block, m):
    pin, sin = _slices(P, m, block, 31 * P + m + block)
    po, so = oracle.qgz_reduce_level(pin, sin, P, m, block)
    gp, gs = zq.qgz_reduce_level(to_dev(pin), to_dev(sin), P, m, block)
    torch.cuda.synchronize()
    assert_bits_equal(from_dev(gp), po, f"reduce packed P={P} B={block} m={m}", block // 2)
    assert_bits_equal(from_dev(gs), so, f"reduce scales P={P} B={block} m={m}")


def test_reduce_identical_and_cancelling():
    m, block = 8192, 128
    g = np.random.default_rng(8)
    x = (g.standard_normal(m) * 1e-3).astype(np.float32)
    p0, s0 = oracle.qgz_quantize(x, block)
    for P in (2, 8, 48):
        gp, gs = zq.qgz_reduce_level(to_dev(np.tile(p0, P)), to_dev(np.tile(s0, P)), P, m, block)
        po, so = oracle.qgz_reduce_level(np.tile(p0, P), np.tile(s0, P), P, m, block)
        torch.cuda.synchronize()
        assert_bits_equal(from_dev(gp), po, f"identical P={P}")
        assert_bits_equal(from_dev(gs), so, f"identical P={P} scales")
    pn, sn = oracle.qgz_quantize(-x, block)
    gp, gs = zq.qgz_reduce_level(to_dev(np.concatenate([p0, pn])), to_dev(np.concatenate([s0, sn])), 2, m, block)
    torch.cuda.synchronize()
    assert not from_dev(gp).any() and not from_dev(gs).any()


def test_three_level_chain_small():
    """The hierarchical chain (fan-ins 2, 4, 48) at a reduced size, composed
    from the C ABI calls, against the oracle's chain."""
    block, fanins, rank = 128, [2, 4, 48], 0
    n = 2 * 4 * 48 * block * 4
    g = np.random.default_rng(12)
    own = (g.standard_normal(n) * 1e-3).astype(np.float32)
    peers, m = [], n
    for k, P in enumerate(fanins):
        m //= P
        lvl = []
        for p in range(P):
            xs = (np.random.default_rng([4, 2, k, p]).standard_normal(m) * 1e-3).astype(np.float32)
            lvl.append(oracle.qgz_quantize(xs, block) if p != rank else None)
        peers.append(lvl)
    op_, os_ = oracle.qgz_quantize(own, block)
    outs = oracle.chain(op_, os_, n, fanins, peers, rank, block)
    want = oracle.qgz_dequantize(outs[-1][0], outs[-1][1], outs[-1][2], block, "f32")

    gp, gs = zq.qgz_quantize(to_dev(own), block)
    cur_m = n
    for k, P in enumerate(fanins):
        m = cur_m // P
        mb, nbm = (m + 1) // 2, m // block
        pin = torch.empty(P * mb, dtype=torch.uint8, device="cuda")
        sin = torch.empty(P * nbm, dtype=torch.float32, device="cuda")
        for p in range(P):
            if p == rank:
                pin[p * mb:(p + 1) * mb] = gp[rank * mb:(rank + 1) * mb]
                sin[p * nbm:(p + 1) * nbm] = gs[rank * nbm:(rank + 1) * nbm]
            else:
                pin[p * mb:(p + 1) * mb] = to_dev(peers[k][p][0])
                sin[p * nbm:(p + 1) * nbm] = to_dev(peers[k][p][1])
        gp, gs = zq.qgz_reduce_level(pin, sin, P, m, block)
        torch.cuda.synchronize()
        assert_bits_equal(from_dev(gp), outs[k][0], f"chain level {k} packed")
        assert_bits_equal(from_dev(gs), outs[k][1], f"chain level {k} scales")
        cur_m = m
    y = zq.qgz_dequantize(gp, gs, cur_m, block, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert_bits_equal(from_dev(y), want, "chain final dequant")


def test_empty_is_noop():
    x = torch.empty(0, device="cuda")
    c, s = zq.qwz_quantize(x, 256)
    assert c.numel() == 0 and s.numel() == 0


def test_async_on_side_stream():
    """Work goes to the given stream; results are complete after syncing it."""
    g = np.random.default_rng(2)
    x = (g.standard_normal(1 << 20) * 1e-3).astype(np.float32)
    want = oracle.qgz_quantize(x, 128)
    s = torch.cuda.Stream()
    xd = to_dev(x)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        gp, gs = zq.qgz_quantize(xd, 128)
    s.synchronize()
    assert_bits_equal(from_dev(gp), want[0], "side stream packed")
    assert_bits_equal(from_dev(gs), want[1], "side stream scales")


def test_argument_error_writes_nothing():
    out = torch.full((256,), 0x5A, dtype=torch.uint8, device="cuda")
    sc = torch.full((4,), 7.0, device="cuda")
    x = torch.ones(512, device="cuda")
    with pytest.raises(zq.ZQError):
        zq.qgz_quantize(x, 48, packed=out, scales=sc)
    torch.cuda.synchronize()
    assert bool((out == 0x5A).all()) and bool((sc == 7.0).all())


FUSED_CASES = [(2, 128, 524288, "f32"), (8, 128, (1 << 23) + 4096, "f32"), (48, 128, 4096 * 32, "f32"),
               (3, 64, 65536 + 64, "bf16"), (4, 256, 8192, "f16"), (8, 128, 1000, "f32"), (2, 1024, 3072, "bf16"),
               (5, 32, 33, "f32"), (2, 128, (1 << 22), "bf16"), (2, 128, (1 << 23) + 4096, "bf16")]


@pytest.mark.parametrize("P,block,m,out", FUSED_CASES)
def test_reduce_dequantize_fused(P, block, m, out):
    """The fused last level equals dequantise(reduce_level(...)) bit for bit,
    with and without the optional INT4 output."""
    pin, sin = _slices(P, m, block, 97 * P + m + block)
    po, so = oracle.qgz_reduce_level(pin, sin, P, m, block)
    want = oracle.qgz_dequantize(po, so, m, block, out)
    dt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[out]
    dpin, dsin = to_dev(pin), to_dev(sin)
    y = zq.qgz_reduce_dequantize(dpin, dsin, P, m, block, out_dtype=dt)
    torch.cuda.synchronize()
    assert_bits_equal(from_dev(y), want, f"fused P={P} B={block} m={m} -> {out}")
    gp = poisoned(zq.int4_bytes(m), torch.uint8)
    gs = poisoned(zq.num_scales(m, block), torch.float32)
    y2 = zq.qgz_reduce_dequantize(dpin, dsin, P, m, block, out_dtype=dt, packed_out=gp, scales_out=gs)
    torch.cuda.synchronize()
    assert_bits_equal(from_dev(y2), want, "fused (with INT4 output)")
    assert_bits_equal(from_dev(gp), po, "fused INT4 packed")
    assert_bits_equal(from_dev(gs), so, "fused INT4 scales")


def test_repeat_runs_bit_identical():
    """Every call is deterministic: two runs give identical bits."""
    g = np.random.default_rng(21)
    n, P, m = (1 << 21) + 1000, 8, 1 << 18
    x = to_dev((g.standard_normal(n) * 1e-3).astype(np.float32))
    pin, sin = _slices(P, m, 128, 5)
    dpin, dsin = to_dev(pin), to_dev(sin)
    outs = []
    for _ in range(2):
        c, s = zq.qwz_quantize(x, 256)
        p4, s4 = zq.qgz_quantize(x, 128)
        rp, rs = zq.qgz_reduce_level(dpin, dsin, P, m, 128)
        y = zq.qgz_reduce_dequantize(dpin, dsin, P, m, 128)
        d8 = zq.qwz_dequantize(c, s, 256, out_dtype=torch.bfloat16)
        torch.cuda.synchronize()
        outs.append([from_dev(t) for t in (c, s, p4, s4, rp, rs, y, d8)])
    for a, b in zip(*outs):
        assert a.tobytes() == b.tobytes()


def test_hip_graph_capture_replays():
    """The entry points enqueue only kernel launches (no allocation, memset or
    synchronisation), so a sequence of calls can be captured in a HIP graph.
    Each replay, with eager work in between, must give the eager bits."""
    g = np.random.default_rng(22)
    n, block = 1 << 20, 128
    x_host = (g.standard_normal(n) * 1e-3).astype(np.float32)
    x = to_dev(x_host)
    P, m = 4, n // 4
    packed = poisoned(n // 2, torch.uint8)
    scales = poisoned(n // block, torch.float32)
    rp = poisoned(m // 2, torch.uint8)
    rs = poisoned(m // block, torch.float32)
    y = poisoned(m, torch.float32)
    yf = poisoned(m, torch.bfloat16)

    def path():
        zq.qgz_quantize(x, block, packed=packed, scales=scales)
        zq.qgz_reduce_level(packed, scales, P, m, block, packed_out=rp, scales_out=rs)
        zq.qgz_dequantize(rp, rs, m, block, y=y)
        zq.qgz_reduce_dequantize(packed, scales, P, m, block, y=yf)

    path()
    torch.cuda.synchronize()
    want = [from_dev(t).copy() for t in (packed, scales, rp, rs, y, yf)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            path()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (packed, scales, rp, rs, y, yf):
            t.zero_()                      # eager work between replays
        graph.replay()
        torch.cuda.synchronize()
        for t, w in zip((packed, scales, rp, rs, y, yf), want):
            assert from_dev(t).tobytes() == w.tobytes(), f"replay {rep}"


def test_concurrent_host_threads_on_separate_streams():
    """The library keeps no state: calls from several host threads, each on its
    own stream (default priority), give the oracle's bits."""
    import threading

    g = np.random.default_rng(23)
    n, block = (1 << 21) + 96, 128
    xs = [(g.standard_normal(n) * 10.0 ** -k).astype(np.float32) for k in range(4)]
    want = [oracle.qgz_quantize(x, block) for x in xs]
    xds = [to_dev(x) for x in xs]
    torch.cuda.synchronize()
    got, errors = [None] * len(xs), []

    def work(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                for _ in range(5):
                    p, sc = zq.qgz_quantize(xds[i], block)
                    y = zq.qgz_dequantize(p, sc, n, block, out_dtype=torch.float32)
            s.synchronize()
            got[i] = (from_dev(p), from_dev(sc), from_dev(y))
        except Exception as e:  # reported below, on the main thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(i,)) for i in range(len(xs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for i, (p, sc, y) in enumerate(got):
        assert_bits_equal(p, want[i][0], f"thread {i} packed", block // 2)
        assert_bits_equal(sc, want[i][1], f"thread {i} scales")
        assert_bits_equal(y, oracle.qgz_dequantize(want[i][0], want[i][1], n, block, "f32"), f"thread {i} dequant")


# Inputs that reach the reduce level's rare branches (tests/pin_checks.py,
# special_reduce_slices): non-zero block sums below the 2^-119 flush
# threshold (with subnormal products), and slice scales above 2^124, for
# which 16 * s is not finite.  Each on the large (P >= 3), two-slice
# (P <= 2) and small-level vector shapes and on the per-block generic kernel
# (ragged m, and the leftover blocks after the last whole group).
SPECIAL_REDUCE_CASES = [
    ("subthreshold", 2, 128, (1 << 23) + 4096),
    ("subthreshold", 3, 128, (1 << 23) + 4096),
    ("subthreshold", 8, 128, 65536 + 128),
    ("subthreshold", 48, 64, 16384),
    ("subthreshold", 5, 64, 4095),
    ("subthreshold", 2, 1024, 16 * 1024 + 32),
    ("huge", 1, 128, (1 << 23) + 4096),
    ("huge", 2, 128, (1 << 23) + 4096),
    ("huge", 3, 128, (1 << 23) + 4096),
    ("huge", 3, 256, 65536 + 256),
    ("huge", 2, 64, 1000),
    # small levels with the slice count fixed at compile time (P = 2, 4, 8)
    ("huge", 2, 128, 65536 + 128),
    ("huge", 4, 64, 32768),
    ("huge", 8, 256, 65536 + 256),
    ("subthreshold", 4, 256, 65536 + 256),
    ("subthreshold", 2, 64, 2048 * 3 + 64),
]


@pytest.mark.parametrize("kind,P,block,m", SPECIAL_REDUCE_CASES)
def test_reduce_edge_sums(kind, P, block, m):
    """The reduce level, the fused last level and the gathered-slice form on
    edge sums, bit for bit against the oracle."""
    what = f"{kind} P={P} B={block} m={m}"
    pin, sin = pc.special_reduce_slices(kind, P, m, block, 7 * P + m + block)
    nb, mb = zq.num_scales(m, block), zq.int4_bytes(m)
    if kind == "subthreshold":
        low, high = pc.subthreshold_block_counts(pin, sin, P, m, block)
        assert low > 0 and high > 0, f"{what}: input misses the flush threshold"
    else:
        assert float(sin[:nb].max()) > 2.0 ** 124, f"{what}: no scale above 2^124"
    po, so = oracle.qgz_reduce_level(pin, sin, P, m, block)
    dpin, dsin = to_dev(pin), to_dev(sin)
    gp, gs = zq.qgz_reduce_level(dpin, dsin, P, m, block)
    torch.cuda.synchronize()
    assert_bits_equal(from_dev(gp), po, f"{what} packed", block // 2)
    assert_bits_equal(from_dev(gs), so, f"{what} scales")
    for out, dt in (("f32", torch.float32), ("bf16", torch.bfloat16)):
        want = oracle.qgz_dequantize(po, so, m, block, out)
        fp, fs = poisoned(mb, torch.uint8), poisoned(nb, torch.float32)
        y = zq.qgz_reduce_dequantize(dpin, dsin, P, m, block, out_dtype=dt, packed_out=fp, scales_out=fs)
        torch.cuda.synchronize()
        assert_bits_equal(from_dev(y), want, f"{what} fused -> {out}")
        assert_bits_equal(from_dev(fp), po, f"{what} fused INT4 packed", block // 2)
        assert_bits_equal(from_dev(fs), so, f"{what} fused INT4 scales")
    ps = [dpin[p * mb:(p + 1) * mb].clone() for p in range(P)]
    ss = [dsin[p * nb:(p + 1) * nb].clone() for p in range(P)]
    hp, hs = zq.qgz_reduce_level_gather(ps, ss, m, block)
    torch.cuda.synchronize()
    assert_bits_equal(from_dev(hp), po, f"{what} gather packed", block // 2)
    assert_bits_equal(from_dev(hs), so, f"{what} gather scales")


# The compile-time-P kernels (P = 2, 4, 8; B = 64, 128, 256): on large levels
# at sizes where the workgroups take T = 4 groups (P = 2) and the group count
# leaves 1, 2 or 3 over, so the last workgroup clamps to the last group and
# recomputes it; on small levels (8 elements per lane, one group per
# workgroup) from one group up.  Some sizes also leave a block for the
# generic kernel.  Plain, fused (f32, bf16) and gathered.
FIXED_P_CASES = [(2, 128, 8192 * 4097), (2, 128, 8192 * 4098 + 128), (2, 256, 8192 * 4099),
                 (2, 64, 8192 * 4097 + 64), (4, 64, 8192 * 4098), (4, 256, 8192 * 4099),
                 (8, 64, 8192 * 4098), (8, 256, 8192 * 4097),
                 # small levels: groups of 2,048 elements, one per workgroup
                 (2, 64, 2048 * 5 + 64), (2, 128, 2048), (2, 256, 2048 * 33 + 512),
                 (4, 64, 2048 * 7), (4, 128, 2048 * 100 + 128), (4, 256, 2048 * 3 + 256),
                 (8, 64, 2048 * 9 + 64), (8, 128, 2048 * 64), (8, 256, 2048 * 11 + 256)]


def _random_level(P, m, block, seed):
    """P slices of random bytes (every nibble value, -8 included; m is even)
    and scales in [1e-4, 1e-3)."""
    assert m % 2 == 0
    g = np.random.default_rng(seed)
    packed = g.integers(0, 256, P * (m // 2), dtype=np.uint8)
    scales = g.uniform(1e-4, 1e-3, P * ((m + block - 1) // block)).astype(np.float32)
    return packed, scales


@pytest.mark.parametrize("P,block,m", FIXED_P_CASES)
def test_reduce_fixed_p_group_tails(P, block, m):
    what = f"P={P} B={block} m={m}"
    pin, sin = _random_level(P, m, block, 13 * P + block + m)
    po, so = oracle.qgz_reduce_level(pin, sin, P, m, block)
    dpin, dsin = to_dev(pin), to_dev(sin)
    nb, mb = zq.num_scales(m, block), zq.int4_bytes(m)
    gp, gs = poisoned(mb, torch.uint8), poisoned(nb, torch.float32)
    zq.qgz_reduce_level(dpin, dsin, P, m, block, packed_out=gp, scales_out=gs)
    torch.cuda.synchronize()
    assert_bits_equal(from_dev(gp), po, f"{what} packed", block // 2)
    assert_bits_equal(from_dev(gs), so, f"{what} scales")
    for out, dt in (("f32", torch.float32), ("bf16", torch.bfloat16)):
        y = zq.qgz_reduce_dequantize(dpin, dsin, P, m, block, out_dtype=dt)
        torch.cuda.synchronize()
        assert_bits_equal(from_dev(y), oracle.qgz_dequantize(po, so, m, block, out), f"{what} fused -> {out}")
    ps = [dpin[p * mb:(p + 1) * mb].clone() for p in range(P)]
    ss = [dsin[p * nb:(p + 1) * nb].clone() for p in range(P)]
    hp, hs = zq.qgz_reduce_level_gather(ps, ss, m, block)
    torch.cuda.synchronize()
    assert_bits_equal(from_dev(hp), po, f"{what} gather packed", block // 2)
    assert_bits_equal(from_dev(hs), so, f"{what} gather scales")
