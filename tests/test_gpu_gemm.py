"""GPU parity of the dequantise-on-load GEMM (qwz_dequant_gemm) with the
oracle.  Two kinds of cases:

* exact: x small multiples of 1/4, scales 2^-7 (so every dequantised weight
  q/128 is exact in bf16 / fp16) -- every partial sum is a multiple of 2^-9
  below 2^15, exact in binary32 in any order, so the result must equal the
  oracle's bit for bit;
* realistic: x ~ N(0, 1), weights N(0, 0.02) quantised by the oracle; the
  binary32 sum in the matrix cores' order is held to
  |y - exact| <= 2 K 2^-24 sum_k |x w| (+ 2^-126 for underflow), the bound for
  any order of K - 1 rounded binary32 additions of exact products.
Plus the layer's four GEMMs (GPT-20B) at 8192 tokens on sampled rows and at
1, 16, 64 and 1024 tokens.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2501_04266_amd as zq
from paper_2501_04266_amd import workloads as wl
from tests.gpu_util import from_dev, poisoned, to_dev

pytestmark = pytest.mark.gpu


def _x_dev(x, dtype):
    return to_dev(x, dtype).reshape(x.shape)


def _exact_inputs(M, N, K, B, dtype, seed):
    rng = np.random.default_rng(seed)
    xf = (rng.integers(-16, 17, (M, K)) / 4.0).astype(np.float32)
    x = wl.to_storage(xf.reshape(-1), dtype).reshape(M, K)
    codes = rng.integers(-127, 128, N * K).astype(np.int8)
    scales = np.full(-(-(N * K) // B), 2.0 ** -7, np.float32)
    return x, codes, scales


# M <= 16: the weight-streaming kernel; 17-128: the ping-pong kernel's
# 128 x 256 tiles; M > 128: its 256 x 256 tiles; K split when the tiles are
# few (down to one K-step per split); ragged edges in M and N and 1, 2, 3
# and 10 K-steps of 64
EXACT = [(1, 1, 64, 256), (37, 100, 192, 32), (17, 70, 320, 64), (40, 300, 1024, 256), (64, 129, 2048, 128),
         (65, 300, 2048, 64), (100, 520, 6144, 256), (127, 257, 192, 32),
         (128, 128, 64, 256), (300, 257, 1024, 128), (129, 383, 640, 64), (256, 512, 6144, 256),
         (600, 300, 64, 256), (513, 257, 128, 64), (777, 520, 192, 32), (1024, 512, 640, 128)]


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("M,N,K,B", EXACT)
def test_dequant_gemm_exact(M, N, K, B, dtype):
    x, codes, scales = _exact_inputs(M, N, K, B, dtype, M * 7 + N + K)
    want = oracle.qwz_dequant_gemm(x, codes, scales, N, B, dtype)
    y = zq.qwz_dequant_gemm(_x_dev(x, dtype), to_dev(codes), to_dev(scales), N, B)
    torch.cuda.synchronize()
    got = from_dev(y).astype(np.float64)
    assert got.shape == (M, N)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} of {got.size} differ; first at {np.unravel_index(bad[0], got.shape)}"


# M <= 16: the weight-streaming kernel (codes straight into the 16 x 16 x 32
# MFMA operands, x staged in LDS over K ranges of up to 1024): ragged N, K
# that ends inside a 256-wide chunk (64, 192, 320, 1088) or inside a
# workgroup's range (4160), one and several ranges per row group, ranges of
# 256, 512 (N = 32768) and 1024 (N = 65600), every block size (B = 32: two
# blocks per 64-code segment)
DECODE = [(1, 1, 64, 32), (2, 70, 192, 64), (7, 129, 320, 128), (15, 1000, 1088, 256), (16, 64, 4160, 1024),
          (16, 4100, 2048, 32), (3, 32768, 960, 512), (16, 65600, 1088, 64)]


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("M,N,K,B", DECODE)
def test_dequant_gemm_decode_exact(M, N, K, B, dtype):
    x, codes, scales = _exact_inputs(M, N, K, B, dtype, 31 * M + N + K)
    want = oracle.qwz_dequant_gemm(x, codes, scales, N, B, dtype)
    y = poisoned(M * N, torch.float32).reshape(M, N)
    zq.qwz_dequant_gemm(_x_dev(x, dtype), to_dev(codes), to_dev(scales), N, B, y=y)
    torch.cuda.synchronize()
    got = from_dev(y).astype(np.float64)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} of {got.size} differ; first at {np.unravel_index(bad[0], got.shape)}"


def _check_bound(got, x, codes, scales, N, B, dtype, what):
    want = oracle.qwz_dequant_gemm(x, codes, scales, N, B, dtype)
    K = x.shape[1]
    wdq = oracle.elements_to_f64(oracle.qwz_dequantize(codes[:N * K], scales, B, dtype), dtype).reshape(N, K)
    mag = np.abs(oracle.elements_to_f64(x, dtype).reshape(x.shape)) @ np.abs(wdq).T
    tol = 2.0 * K * 2.0 ** -24 * mag + 2.0 ** -126
    err = np.abs(got.astype(np.float64) - want)
    worst = np.unravel_index(np.argmax(err - tol), err.shape)
    assert np.all(err <= tol), f"{what}: error {err[worst]:.3e} > bound {tol[worst]:.3e} at {worst}"
    return float((err / np.maximum(mag, 1e-300)).max())


# M <= 16 the weight-streaming kernel, 17-128 the 128 x 256 tiles, larger M
# the 256 x 256 tiles; all but (1, 128, 64, 32) split K across workgroups
REAL = [(256, 384, 6144, 256), (100, 130, 1024, 64), (64, 256, 24576, 256), (1, 128, 64, 32),
        (16, 24576, 6144, 256), (200, 6144, 24576, 256), (257, 640, 1024, 128), (513, 256, 1024, 256)]


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("M,N,K,B", REAL)
def test_dequant_gemm_realistic(M, N, K, B, dtype):
    xf = wl.normal_f32(M * K, 1.0, key=[8, wl.ROLE_MISC, M, K])
    x = wl.to_storage(xf, dtype).reshape(M, K)
    w = wl.weights(N * K, "f32", key=[8, wl.ROLE_WEIGHT, N, K])
    codes, scales = oracle.qwz_quantize(w, B, "f32")
    y = zq.qwz_dequant_gemm(_x_dev(x, dtype), to_dev(codes), to_dev(scales), N, B)
    torch.cuda.synchronize()
    _check_bound(from_dev(y), x, codes, scales, N, B, dtype, f"M={M} N={N} K={K} B={B} {dtype}")


@pytest.mark.parametrize("shift", [1, 2, 3])
@pytest.mark.parametrize("M,N,K", [(5, 70, 320), (40, 100, 1024), (600, 300, 12288)])
def test_dequant_gemm_split_y_not_16_byte_aligned(M, N, K, shift):
    """Split launches first zero y, then add partial tiles into it; y placed
    4, 8 or 12 bytes past a 16-byte boundary (the C ABI asks only 4-byte
    alignment of y), inside a poisoned buffer: the result is exact and no
    float outside y changes.
    (5, 70, 320) splits K on the weight-streaming path, (40, 100, 1024) on
    the 128 x 256 tiles, (600, 300, 12288) on the 256 x 256 tiles."""
    x, codes, scales = _exact_inputs(M, N, K, 256, "bf16", 4 * M + shift)
    want = oracle.qwz_dequant_gemm(x, codes, scales, N, 256, "bf16")
    buf = poisoned(M * N + 8, torch.float32)
    guard = buf.clone()
    y = buf[shift:shift + M * N].view(M, N)
    assert y.data_ptr() % 16 == 4 * shift
    zq.qwz_dequant_gemm(_x_dev(x, "bf16"), to_dev(codes), to_dev(scales), N, 256, y=y)
    torch.cuda.synchronize()
    got = from_dev(y).astype(np.float64)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} of {got.size} differ; first at {np.unravel_index(bad[0], got.shape)}"
    outside = torch.cat([buf[:shift], buf[shift + M * N:]]).view(torch.int32)
    assert torch.equal(outside, torch.cat([guard[:shift], guard[shift + M * N:]]).view(torch.int32))


def test_dequant_gemm_k_zero_and_empty():
    x = torch.zeros((5, 0), dtype=torch.bfloat16, device="cuda")
    codes = torch.zeros(16, dtype=torch.int8, device="cuda")
    scales = torch.zeros(1, dtype=torch.float32, device="cuda")
    y = poisoned(5 * 7, torch.float32).reshape(5, 7)
    zq.qwz_dequant_gemm(x, codes, scales, 7, 256, y=y)
    torch.cuda.synchronize()
    assert bool((y == 0).all())
    x0 = torch.zeros((0, 64), dtype=torch.bfloat16, device="cuda")
    assert zq.qwz_dequant_gemm(x0, codes, scales, 0, 256).shape == (0, 0)


def test_dequant_gemm_rejects_ragged_k():
    x = torch.zeros((4, 96), dtype=torch.bfloat16, device="cuda")
    codes = torch.zeros(4 * 96, dtype=torch.int8, device="cuda")
    scales = torch.zeros(2, dtype=torch.float32, device="cuda")
    with pytest.raises(zq.ZQError):
        zq.qwz_dequant_gemm(x, codes, scales, 4, 256)


@pytest.fixture(scope="module")
def gpt20b_layer():
    """The gathered INT8 GPT-20B layer (oracle-quantised once for the module),
    on the host and on the device."""
    w = wl.weights(wl.N_20B, "bf16", key=[3, wl.ROLE_WEIGHT, 0, 0])
    codes, scales = oracle.qwz_quantize(w, 256, "bf16")
    del w
    return codes, scales, to_dev(codes), to_dev(scales)


def _layer_gemms(layer, M, rows):
    """The four forward GEMMs of the GPT-20B layer (QKV 3h x h, attention out
    h x h, FC1 4h x h, FC2 h x 4h; h = 6144) over M tokens, weights taken from
    the gathered INT8 layer at their offsets; the given rows of each output
    against the oracle, within the binary32 accumulation bound."""
    codes, scales, dcodes, dscales = layer
    h, B = 6144, 256
    off = 0
    for name, N, K in (("qkv", 3 * h, h), ("attn_out", h, h), ("fc1", 4 * h, h), ("fc2", h, 4 * h)):
        xf = wl.normal_f32(M * K, 1.0, key=[8, wl.ROLE_MISC, 1, K])
        x = wl.to_storage(xf, "bf16").reshape(M, K)
        y = zq.qwz_dequant_gemm(_x_dev(x, "bf16"), dcodes[off:off + N * K], dscales[off // B:(off + N * K) // B],
                                N, B)
        torch.cuda.synchronize()
        got = from_dev(y[torch.from_numpy(rows).cuda()])
        _check_bound(got, x[rows], codes[off:off + N * K], scales[off // B:(off + N * K) // B], N, B, "bf16",
                     f"{name} M={M}")
        off += N * K


def test_gpt20b_layer_gemms_sampled_rows(gpt20b_layer):
    """The layer's four GEMMs over 8192 tokens (the launch configuration the
    bench times): 24 sampled rows of each output."""
    M = 8192
    _layer_gemms(gpt20b_layer, M, np.unique(np.concatenate([[0, M - 1], np.random.default_rng(9).integers(0, M, 22)])))


@pytest.mark.parametrize("M", [1, 16, 64, 1024])
def test_gpt20b_layer_gemms_few_tokens(gpt20b_layer, M):
    """The same four GEMMs at the token counts of the other kernel paths: the
    weight-streaming kernel (1, 16), the 128 x 256 tiles with K split (64),
    the 256 x 256 tiles, split for attention output and FC2 (1024).  Every
    row up to 32 tokens, else 24 sampled rows."""
    rows = np.arange(M) if M <= 32 else np.unique(
        np.concatenate([[0, M - 1], np.random.default_rng(M).integers(0, M, 22)]))
    _layer_gemms(gpt20b_layer, M, rows)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("M,N,K,B", [(600, 300, 12288, 256), (700, 300, 24576, 128)])
def test_dequant_gemm_large_tiles_split_k(M, N, K, B, dtype):
    """Few 256 x 256 tiles with a long K: the host splits K across workgroups
    (16 ways here) that add their partial tiles into a zeroed y.  x = a/4
    with |a| <= 4 keeps every partial sum a multiple of 2^-9 below 2^15, so
    the result is exact in any order of the additions."""
    rng = np.random.default_rng(M + K)
    x = wl.to_storage((rng.integers(-4, 5, M * K) / 4.0).astype(np.float32), dtype).reshape(M, K)
    codes = rng.integers(-127, 128, N * K).astype(np.int8)
    scales = np.full(-(-(N * K) // B), 2.0 ** -7, np.float32)
    want = oracle.qwz_dequant_gemm(x, codes, scales, N, B, dtype)
    y = zq.qwz_dequant_gemm(_x_dev(x, dtype), to_dev(codes), to_dev(scales), N, B)
    torch.cuda.synchronize()
    got = from_dev(y).astype(np.float64)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} of {got.size} differ; first at {np.unravel_index(bad[0], got.shape)}"


@pytest.mark.parametrize("K", [1 << 21, (1 << 21) + 256])
def test_dequant_gemm_long_k(K):
    """Reductions as long as 2^21 take the ping-pong schedule (32-bit lane
    offsets); longer ones the plain 256 x 256 schedule (64-bit addresses).
    x is zero outside two 4096-column windows at the start and the end of K,
    so the result equals the oracle's GEMM over those columns alone (zero
    terms add exactly); x = a/4 with |a| <= 8 and scales 2^-7 keep every
    partial sum a multiple of 2^-9 below 2^14, exact in binary32."""
    M, N, B, W = 513, 3, 256, 4096
    rng = np.random.default_rng(K % 1000)
    xs = wl.to_storage((rng.integers(-8, 9, (M, 2 * W)) / 4.0).astype(np.float32).reshape(-1), "bf16").reshape(M, 2 * W)
    codes = rng.integers(-127, 128, N * K).astype(np.int8)
    scales = np.full(N * K // B, 2.0 ** -7, np.float32)
    xd = torch.zeros((M, K), dtype=torch.bfloat16, device="cuda")
    xd[:, :W] = to_dev(np.ascontiguousarray(xs[:, :W]), "bf16")
    xd[:, K - W:] = to_dev(np.ascontiguousarray(xs[:, W:]), "bf16")
    y = zq.qwz_dequant_gemm(xd, to_dev(codes), to_dev(scales), N, B)
    torch.cuda.synchronize()
    cw = codes.reshape(N, K)
    sub_codes = np.ascontiguousarray(np.concatenate([cw[:, :W], cw[:, K - W:]], axis=1)).reshape(-1)
    sub_scales = np.full(N * 2 * W // B, 2.0 ** -7, np.float32)
    want = oracle.qwz_dequant_gemm(xs, sub_codes, sub_scales, N, B, "bf16")
    got = from_dev(y).astype(np.float64)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} of {got.size} differ; first at {np.unravel_index(bad[0], got.shape)}"


@pytest.mark.parametrize("M", [8, 64, 640])
def test_dequant_gemm_graph_capture(M):
    """The GEMM only enqueues kernels, so it replays from a HIP graph: the
    weight-streaming path (M = 8) and the 128 x 256 tiles (M = 64), both
    split (each also launches its own zero fill), and the 256 x 256 tiles
    (M = 640); exact inputs make every replay bit-identical."""
    N, K, B = 384, 2048, 256
    x, codes, scales = _exact_inputs(M, N, K, B, "bf16", 31 + M)
    xd, cd, sd = _x_dev(x, "bf16"), to_dev(codes), to_dev(scales)
    y = poisoned(M * N, torch.float32).reshape(M, N)
    want = oracle.qwz_dequant_gemm(x, codes, scales, N, B, "bf16")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            zq.qwz_dequant_gemm(xd, cd, sd, N, B, y=y)
    torch.cuda.synchronize()
    for rep in range(3):
        y.fill_(float("nan"))          # eager work between replays
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(from_dev(y).astype(np.float64), want), f"replay {rep}"
