"""CPU oracle of the qwZ / qgZ compression path -- TEST INFRASTRUCTURE ONLY.

Only tests/, the smoke check in __graft_entry__ and the CPU-baseline leg of
bench.py may import this package.  The product path (the HIP library behind
include/zq.h) never imports it and never falls back to it.

Thin numpy/ctypes wrappers around oracle/zq_oracle.c.  Element arrays are
numpy arrays: float32, float16, or uint16 holding bfloat16 bit patterns
(pass dtype="bf16" for those).  The method, and every reading taken where the
paper is silent, is documented in zq_oracle.c.

`qwz_dequant_gemm` is the forward product of a layer whose weight is held as
the gathered INT8 buffer: dequantise (this package's qwz_dequantize), then one
float64 matrix product.

The 3-level chain (`chain`) composes reduce levels the way the paper's
hierarchical partitioning stacks them (Design: weights over a GCD pair,
gradients over a node, optimizer states over all ranks): level k receives P_k
slices of m_k = m_{k-1} / P_k elements; the local slice is chunk r of the
previous level's output.
"""
import ctypes
import os

import numpy as np

from . import build as _build

DT = {"f32": 0, "f16": 1, "bf16": 2}
_NP = {"f32": np.float32, "f16": np.float16, "bf16": np.uint16}
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = os.environ.get("ZQ_ORACLE_LIB")   # tests load deliberately broken copies this way
    if not path:
        path = _build.LIB
        if not os.path.exists(path):
            _build.build()
    lib = ctypes.CDLL(path)
    i64, i32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
    for name, args in {
        "zqo_qwz_quantize": [vp, ctypes.c_int, i64, i32, vp, vp],
        "zqo_qwz_dequantize": [vp, vp, i64, i32, vp, ctypes.c_int],
        "zqo_qgz_quantize": [vp, ctypes.c_int, i64, i32, vp, vp],
        "zqo_qgz_dequantize": [vp, vp, i64, i32, vp, ctypes.c_int],
        "zqo_qgz_reduce_level": [vp, vp, i32, i64, i32, vp, vp],
    }.items():
        fn = getattr(lib, name)
        fn.argtypes, fn.restype = args, ctypes.c_int
    lib.zqo_set_threads.argtypes, lib.zqo_set_threads.restype = [ctypes.c_int], None
    lib.zqo_get_threads.argtypes, lib.zqo_get_threads.restype = [], ctypes.c_int
    lib.zqo_f32_to_f16.argtypes, lib.zqo_f32_to_f16.restype = [ctypes.c_float], ctypes.c_uint16
    lib.zqo_f32_to_bf16.argtypes, lib.zqo_f32_to_bf16.restype = [ctypes.c_float], ctypes.c_uint16
    lib.zqo_f16_to_f32.argtypes, lib.zqo_f16_to_f32.restype = [ctypes.c_uint16], ctypes.c_float
    _lib = lib
    return lib


class OracleError(RuntimeError):
    pass


def _check(st, what):
    if st != 0:
        raise OracleError(f"{what}: oracle status {st}")


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _elem(x, dtype):
    x = np.ascontiguousarray(x)
    if x.dtype != _NP[dtype]:
        raise TypeError(f"dtype {dtype} wants numpy {_NP[dtype].__name__}, got {x.dtype}")
    return x


def num_scales(n, block):
    return (n + block - 1) // block


def int4_bytes(n):
    return (n + 1) // 2


def set_threads(t):
    _load().zqo_set_threads(int(t))


def get_threads():
    return _load().zqo_get_threads()


def qwz_quantize(x, block, dtype="f32"):
    """INT8 block quantisation -> (codes int8[n], scales float32[ceil(n/B)])."""
    lib = _load()
    x = _elem(x, dtype)
    n = x.size
    codes = np.empty(n, np.int8)
    scales = np.empty(num_scales(n, block), np.float32)
    _check(lib.zqo_qwz_quantize(_ptr(x), DT[dtype], n, block, _ptr(codes), _ptr(scales)), "qwz_quantize")
    return codes, scales


def qwz_dequantize(codes, scales, block, out_dtype="f32"):
    lib = _load()
    codes = np.ascontiguousarray(codes, np.int8)
    scales = np.ascontiguousarray(scales, np.float32)
    n = codes.size
    if scales.size < num_scales(n, block):
        raise ValueError("too few scales")
    y = np.empty(n, _NP[out_dtype])
    _check(lib.zqo_qwz_dequantize(_ptr(codes), _ptr(scales), n, block, _ptr(y), DT[out_dtype]), "qwz_dequantize")
    return y


def qgz_quantize(g, block, dtype="f32"):
    """INT4 block quantisation -> (packed uint8[ceil(n/2)], scales float32[ceil(n/B)])."""
    lib = _load()
    g = _elem(g, dtype)
    n = g.size
    packed = np.empty(int4_bytes(n), np.uint8)
    scales = np.empty(num_scales(n, block), np.float32)
    _check(lib.zqo_qgz_quantize(_ptr(g), DT[dtype], n, block, _ptr(packed), _ptr(scales)), "qgz_quantize")
    return packed, scales


def qgz_dequantize(packed, scales, n, block, out_dtype="f32"):
    lib = _load()
    packed = np.ascontiguousarray(packed, np.uint8)
    scales = np.ascontiguousarray(scales, np.float32)
    if packed.size < int4_bytes(n) or scales.size < num_scales(n, block):
        raise ValueError("input too short")
    y = np.empty(n, _NP[out_dtype])
    _check(lib.zqo_qgz_dequantize(_ptr(packed), _ptr(scales), n, block, _ptr(y), DT[out_dtype]), "qgz_dequantize")
    return y


def qgz_reduce_level(packed_in, scales_in, P, m, block):
    """Dequant -> sum over P slices -> INT4 requant.  packed_in is [P, ceil(m/2)]
    (or flat), scales_in is [P, ceil(m/B)] (or flat)."""
    lib = _load()
    packed_in = np.ascontiguousarray(packed_in, np.uint8).reshape(-1)
    scales_in = np.ascontiguousarray(scales_in, np.float32).reshape(-1)
    if packed_in.size != P * int4_bytes(m) or scales_in.size != P * num_scales(m, block):
        raise ValueError("slice buffer size does not match P, m, block")
    out = np.empty(int4_bytes(m), np.uint8)
    sc = np.empty(num_scales(m, block), np.float32)
    _check(lib.zqo_qgz_reduce_level(_ptr(packed_in), _ptr(scales_in), P, m, block, _ptr(out), _ptr(sc)),
           "qgz_reduce_level")
    return out, sc


def chain(own_packed, own_scales, n, fanins, peer_slices, rank, block):
    """Multi-level qgZ reduction (a stack of reduce levels).

    own_packed/own_scales: INT4 quantisation of this rank's n-element gradient.
    fanins: [P_1, P_2, ...]; level k splits the previous output of m_{k-1}
    elements into P_k chunks of m_k = m_{k-1} / P_k and keeps chunk `rank`.
    peer_slices[k]: list of P_k (packed, scales) pairs for that level, with the
    entry at index `rank` ignored (the local chunk is used instead).
    Returns the list of per-level outputs [(packed, scales, m_k), ...].
    """
    outs = []
    cur_p, cur_s, cur_m = own_packed, own_scales, n
    for k, P in enumerate(fanins):
        if cur_m % P:
            raise ValueError("level size not divisible by fan-in")
        m = cur_m // P
        if m % block:
            raise ValueError("chunk not block aligned")
        nbm, mb = num_scales(m, block), int4_bytes(m)
        own_chunk_p = cur_p[rank * mb:(rank + 1) * mb]
        own_chunk_s = cur_s[rank * nbm:(rank + 1) * nbm]
        slices_p, slices_s = [], []
        for p in range(P):
            if p == rank:
                slices_p.append(own_chunk_p)
                slices_s.append(own_chunk_s)
            else:
                slices_p.append(peer_slices[k][p][0])
                slices_s.append(peer_slices[k][p][1])
        cur_p, cur_s = qgz_reduce_level(np.concatenate(slices_p), np.concatenate(slices_s), P, m, block)
        cur_m = m
        outs.append((cur_p, cur_s, m))
    return outs


def f32_to_f16_bits(v):
    return _load().zqo_f32_to_f16(float(v))


def f32_to_bf16_bits(v):
    return _load().zqo_f32_to_bf16(float(v))


def f16_bits_to_f32(h):
    return _load().zqo_f16_to_f32(int(h))


def elements_to_f64(a, dtype):
    """float32 / float16 arrays, or uint16 bfloat16 bit patterns, widened to
    float64 exactly."""
    if dtype == "bf16":
        return (np.asarray(a, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(a).astype(np.float64)


def qwz_dequant_gemm(x, codes, scales, N, block, dtype="bf16"):
    """Forward product of a layer whose weight arrives as the gathered INT8
    buffer (Design, Weight Partitioning: the Allgathered weight is dequantised
    for the forward pass): y = x @ W^T.  W is the N x K weight in PyTorch Linear
    layout, W[n][k] = element n*K + k of qwz_dequantize(codes, scales, block,
    dtype); x is [M, K] of dtype (bf16 as uint16 bit patterns).  Returns y as
    float64 [M, N].

    The steps are the definition as written: dequantise, then one float64
    matrix product.  Each product of two bf16 / fp16 values is exact in
    float64; the float64 sum is within K * 2^-53 * sum_k |x w| of the exact
    value, far inside the binary32-accumulation bound (2 K 2^-24 sum_k |x w|)
    a GPU result is held to."""
    x = np.asarray(x)
    M, K = x.shape
    w = qwz_dequantize(np.asarray(codes)[:N * K], scales, block, dtype)
    W = elements_to_f64(w, dtype).reshape(N, K)
    X = elements_to_f64(x, dtype).reshape(M, K)
    return X @ W.T
