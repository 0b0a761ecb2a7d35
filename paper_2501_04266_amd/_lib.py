"""ctypes binding of libzq.so (include/zq.h).

Argument marshalling only: every step runs in the HIP kernels.  Tensors are
torch tensors on the GPU (torch is used for device memory and streams); the
work is enqueued on torch's current stream unless `stream` is given.  There is
no CPU fallback: if the library is not built this module raises on use.
"""
import ctypes
import os

import torch  # noqa: F401  -- loads torch's HIP runtime first, so libzq binds to the same one

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("ZQ_LIBRARY") or os.path.join(_PKG, "libzq.so")

ZQ_F32, ZQ_F16, ZQ_BF16 = 0, 1, 2
STATUS = {0: "ZQ_OK", -1: "ZQ_E_NULL", -2: "ZQ_E_BLOCK", -3: "ZQ_E_DTYPE", -4: "ZQ_E_ALIGN",
          -5: "ZQ_E_SIZE", -6: "ZQ_E_P", -7: "ZQ_E_HIP", -8: "ZQ_E_ALIAS"}
EXPORTS = ["qwz_quantize", "qwz_dequantize", "qgz_quantize", "qgz_reduce_level", "qgz_dequantize",
           "qgz_reduce_dequantize", "qgz_reduce_level_gather", "qgz_reduce_level_gather_noalloc",
           "qwz_dequant_gemm", "zq_num_scales", "zq_int4_bytes", "zq_status_string"]

_TORCH_DT = {torch.float32: ZQ_F32, torch.float16: ZQ_F16, torch.bfloat16: ZQ_BF16}
_DT_TORCH = {v: k for k, v in _TORCH_DT.items()}
_lib = None


class ZQError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {STATUS.get(status, status)} ({lib().zq_status_string(status).decode()})")


def lib():
    """The loaded libzq.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2501_04266_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, i32, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int
    sig = {
        "qwz_quantize": [vp, ci, i64, i32, vp, vp, vp],
        "qwz_dequantize": [vp, vp, i64, i32, vp, ci, vp],
        "qgz_quantize": [vp, ci, i64, i32, vp, vp, vp],
        "qgz_dequantize": [vp, vp, i64, i32, vp, ci, vp],
        "qgz_reduce_level": [vp, vp, i32, i64, i32, vp, vp, vp],
        "qgz_reduce_dequantize": [vp, vp, i32, i64, i32, vp, ci, vp, vp, vp],
        "qwz_dequant_gemm": [vp, ci, vp, vp, i64, i64, i64, i32, vp, vp],
        "qgz_reduce_level_gather": [vp, vp, i32, i64, i32, vp, vp, vp],
        "qgz_reduce_level_gather_noalloc": [vp, vp, i32, i64, i32, vp, vp, vp],
    }
    for name, args in sig.items():
        fn = getattr(L, name)
        fn.argtypes, fn.restype = args, ci
    L.zq_num_scales.argtypes, L.zq_num_scales.restype = [i64, i32], i64
    L.zq_int4_bytes.argtypes, L.zq_int4_bytes.restype = [i64], i64
    L.zq_status_string.argtypes, L.zq_status_string.restype = [ci], ctypes.c_char_p
    _lib = L
    return L


def num_scales(n, block):
    return (n + block - 1) // block


def int4_bytes(n):
    return (n + 1) // 2


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dev(t, name):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _need(t, name, count, dtypes):
    """Host-side size and dtype check of a caller's buffer: the C ABI takes raw
    pointers and cannot tell an undersized buffer from a large one."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}; expected one of {[str(d) for d in dtypes]}")
    if t.numel() < count:
        raise ValueError(f"{name} holds {t.numel()} elements; {count} needed")


def _nsc(n, block):
    """Scales needed for n elements; 0 for a block the library will reject
    itself (ZQ_E_BLOCK), so that error is reported as the library's."""
    if not isinstance(block, int) or block < 32 or block > 1024 or block & (block - 1):
        return 0
    return num_scales(n, block)


def _alloc_nsc(n, block):
    """Scales to allocate for n elements (one for a block the library rejects)."""
    return _nsc(n, block) if _nsc(n, block) or n == 0 else 1


_ELEM = (torch.float32, torch.float16, torch.bfloat16)
_I8 = (torch.int8,)
_U8 = (torch.uint8,)
_F32 = (torch.float32,)


def _check(status, what):
    if status != 0:
        raise ZQError(status, what)


def qwz_quantize(x, block=256, codes=None, scales=None, stream=None):
    """INT8 block quantisation of x (f32/f16/bf16) -> (codes int8[n], scales f32[ceil(n/B)])."""
    n = x.numel()
    _need(x, "x", n, _ELEM)
    if codes is None:
        codes = torch.empty(n, dtype=torch.int8, device=x.device)
    if scales is None:
        scales = torch.empty(_alloc_nsc(n, block), dtype=torch.float32, device=x.device)
    _need(codes, "codes", n, _I8)
    _need(scales, "scales", _nsc(n, block), _F32)
    _check(lib().qwz_quantize(_dev(x, "x"), _TORCH_DT[x.dtype], n, block, _dev(codes, "codes"),
                              _dev(scales, "scales"), _stream(stream)), "qwz_quantize")
    return codes, scales


def qwz_dequantize(codes, scales, block=256, out_dtype=torch.bfloat16, y=None, n=None, stream=None):
    n = codes.numel() if n is None else n
    if y is None:
        y = torch.empty(n, dtype=out_dtype, device=codes.device)
    _need(codes, "codes", n, _I8)
    _need(scales, "scales", _nsc(n, block), _F32)
    _need(y, "y", n, _ELEM)
    _check(lib().qwz_dequantize(_dev(codes, "codes"), _dev(scales, "scales"), n, block, _dev(y, "y"),
                                _TORCH_DT[y.dtype], _stream(stream)), "qwz_dequantize")
    return y


def qgz_quantize(g, block=128, packed=None, scales=None, stream=None):
    """INT4 block quantisation -> (packed uint8[ceil(n/2)], scales f32[ceil(n/B)])."""
    n = g.numel()
    _need(g, "g", n, _ELEM)
    if packed is None:
        packed = torch.empty(int4_bytes(n), dtype=torch.uint8, device=g.device)
    if scales is None:
        scales = torch.empty(_alloc_nsc(n, block), dtype=torch.float32, device=g.device)
    _need(packed, "packed", int4_bytes(n), _U8)
    _need(scales, "scales", _nsc(n, block), _F32)
    _check(lib().qgz_quantize(_dev(g, "g"), _TORCH_DT[g.dtype], n, block, _dev(packed, "packed"),
                              _dev(scales, "scales"), _stream(stream)), "qgz_quantize")
    return packed, scales


def qgz_dequantize(packed, scales, n, block=128, out_dtype=torch.float32, y=None, stream=None):
    if y is None:
        y = torch.empty(n, dtype=out_dtype, device=packed.device)
    _need(packed, "packed", int4_bytes(n), _U8)
    _need(scales, "scales", _nsc(n, block), _F32)
    _need(y, "y", n, _ELEM)
    _check(lib().qgz_dequantize(_dev(packed, "packed"), _dev(scales, "scales"), n, block, _dev(y, "y"),
                                _TORCH_DT[y.dtype], _stream(stream)), "qgz_dequantize")
    return y


def qgz_reduce_level(packed_in, scales_in, P, m, block=128, packed_out=None, scales_out=None, stream=None):
    """Dequant -> sum over P slices (ascending) -> INT4 requant.  packed_in holds
    P slices of ceil(m/2) bytes back to back, scales_in P x ceil(m/B)."""
    dev = packed_in.device
    if packed_out is None:
        packed_out = torch.empty(int4_bytes(m), dtype=torch.uint8, device=dev)
    if scales_out is None:
        scales_out = torch.empty(_alloc_nsc(m, block), dtype=torch.float32, device=dev)
    _need(packed_in, "packed_in", P * int4_bytes(m), _U8)
    _need(scales_in, "scales_in", P * _nsc(m, block), _F32)
    _need(packed_out, "packed_out", int4_bytes(m), _U8)
    _need(scales_out, "scales_out", _nsc(m, block), _F32)
    _check(lib().qgz_reduce_level(_dev(packed_in, "packed_in"), _dev(scales_in, "scales_in"), P, m, block,
                                  _dev(packed_out, "packed_out"), _dev(scales_out, "scales_out"),
                                  _stream(stream)), "qgz_reduce_level")
    return packed_out, scales_out


def qgz_reduce_dequantize(packed_in, scales_in, P, m, block=128, out_dtype=torch.float32, y=None,
                          packed_out=None, scales_out=None, stream=None):
    """Last level fused with the final dequantisation: returns y (m elements of
    out_dtype) bit-identical to qgz_dequantize(qgz_reduce_level(...)).  Pass
    packed_out and scales_out to also receive the INT4 result."""
    if y is None:
        y = torch.empty(m, dtype=out_dtype, device=packed_in.device)
    if (packed_out is None) != (scales_out is None):
        raise ValueError("give both packed_out and scales_out, or neither")
    _need(packed_in, "packed_in", P * int4_bytes(m), _U8)
    _need(scales_in, "scales_in", P * _nsc(m, block), _F32)
    _need(y, "y", m, _ELEM)
    if packed_out is not None:
        _need(packed_out, "packed_out", int4_bytes(m), _U8)
        _need(scales_out, "scales_out", _nsc(m, block), _F32)
    _check(lib().qgz_reduce_dequantize(_dev(packed_in, "packed_in"), _dev(scales_in, "scales_in"), P, m, block,
                                       _dev(y, "y"), _TORCH_DT[y.dtype],
                                       None if packed_out is None else _dev(packed_out, "packed_out"),
                                       None if scales_out is None else _dev(scales_out, "scales_out"),
                                       _stream(stream)), "qgz_reduce_dequantize")
    return y


def gather_tables(packed_slices, scale_slices):
    """Device tables (int64 tensors) of the slices' addresses, for
    qgz_reduce_level_gather; build them once to reuse them, e.g. under graph
    capture, where the per-call host-to-device copy is not allowed."""
    dev = packed_slices[0].device
    tab = torch.tensor([_dev(t, "packed_slices[p]") for t in packed_slices], dtype=torch.int64).to(dev)
    stab = torch.tensor([_dev(t, "scale_slices[p]") for t in scale_slices], dtype=torch.int64).to(dev)
    return tab, stab


def qgz_reduce_level_gather(packed_slices, scale_slices, m, block=128, packed_out=None, scales_out=None,
                            stream=None, tables=None):
    """qgz_reduce_level over P slices held in separate tensors (lists of P
    uint8 tensors of ceil(m/2) bytes and P float32 tensors of ceil(m/B)
    scales), read in place through device tables of their addresses (built
    here, or passed as `tables` from gather_tables).  Bit-identical to
    qgz_reduce_level on the slices laid out back to back."""
    P = len(packed_slices)
    if P != len(scale_slices) or P == 0:
        raise ValueError("give P >= 1 byte slices and as many scale slices")
    for p, (a, b) in enumerate(zip(packed_slices, scale_slices)):
        _need(a, f"packed_slices[{p}]", int4_bytes(m), _U8)
        _need(b, f"scale_slices[{p}]", _nsc(m, block), _F32)
        # the library reads the slice addresses on the device and cannot check
        # them itself: the vector path (m % 32 == 0) loads 16 bytes per lane
        if m % 32 == 0 and _dev(a, f"packed_slices[{p}]") % 16:
            raise ValueError(f"packed_slices[{p}] must be 16-byte aligned when m % 32 == 0")
        if _dev(b, f"scale_slices[{p}]") % 4:
            raise ValueError(f"scale_slices[{p}] must be 4-byte aligned")
    dev = packed_slices[0].device
    if packed_out is None:
        packed_out = torch.empty(int4_bytes(m), dtype=torch.uint8, device=dev)
    if scales_out is None:
        scales_out = torch.empty(_alloc_nsc(m, block), dtype=torch.float32, device=dev)
    _need(packed_out, "packed_out", int4_bytes(m), _U8)
    _need(scales_out, "scales_out", _nsc(m, block), _F32)
    # the pointer tables live in device memory (the kernel reads them); built
    # here they are allocated on the current stream and, if the call runs on
    # another (a torch stream or a raw handle), recorded on it so the
    # allocator keeps them until the kernel has read them
    if tables is None:
        tab, stab = gather_tables(packed_slices, scale_slices)
        if stream is not None:
            st = stream if hasattr(stream, "cuda_stream") else torch.cuda.ExternalStream(int(stream))
            tab.record_stream(st)
            stab.record_stream(st)
    else:
        tab, stab = tables
        _need(tab, "tables[0]", P, (torch.int64,))
        _need(stab, "tables[1]", P, (torch.int64,))
    _check(lib().qgz_reduce_level_gather(tab.data_ptr(), stab.data_ptr(), P, m, block,
                                         _dev(packed_out, "packed_out"), _dev(scales_out, "scales_out"),
                                         _stream(stream)), "qgz_reduce_level_gather")
    return packed_out, scales_out


def qgz_reduce_level_gather_noalloc(packed_slices, scale_slices, m, block, packed_out, scales_out, stream=None):
    """qgz_reduce_level_gather without any device allocation: the slice
    addresses go to the library in host arrays (it keeps its own device table
    per GPU), and the caller passes the outputs.  Calls that may overlap on
    one GPU share that table and must be ordered (one stream)."""
    import ctypes
    P = len(packed_slices)
    if P != len(scale_slices) or P == 0:
        raise ValueError("give P >= 1 byte slices and as many scale slices")
    for p, (a, b) in enumerate(zip(packed_slices, scale_slices)):
        _need(a, f"packed_slices[{p}]", int4_bytes(m), _U8)
        _need(b, f"scale_slices[{p}]", _nsc(m, block), _F32)
    _need(packed_out, "packed_out", int4_bytes(m), _U8)
    _need(scales_out, "scales_out", _nsc(m, block), _F32)
    tab = (ctypes.c_void_p * P)(*[_dev(t, f"packed_slices[{p}]") for p, t in enumerate(packed_slices)])
    stab = (ctypes.c_void_p * P)(*[_dev(t, f"scale_slices[{p}]") for p, t in enumerate(scale_slices)])
    _check(lib().qgz_reduce_level_gather_noalloc(ctypes.cast(tab, ctypes.c_void_p), ctypes.cast(stab, ctypes.c_void_p),
                                                 P, m, block, _dev(packed_out, "packed_out"),
                                                 _dev(scales_out, "scales_out"), _stream(stream)),
           "qgz_reduce_level_gather_noalloc")
    return packed_out, scales_out


def qwz_dequant_gemm(x, codes, scales, N, block=256, y=None, stream=None):
    """y[M, N] = x[M, K] @ deq(W)^T with W the N x K INT8 weight (codes int8
    [N*K] row-major, scales [ceil(N*K/block)]) dequantised to x's dtype
    (bf16 or fp16) on load; y is float32.  K must be a multiple of 64."""
    if x.dim() != 2:
        raise ValueError("x must be 2-D [M, K]")
    M, K = x.shape
    _need(x, "x", M * K, (torch.bfloat16, torch.float16))
    _need(codes, "codes", N * K, _I8)
    _need(scales, "scales", _nsc(N * K, block), _F32)
    if y is None:
        y = torch.empty((M, N), dtype=torch.float32, device=x.device)
    _need(y, "y", M * N, _F32)
    _check(lib().qwz_dequant_gemm(_dev(x, "x"), _TORCH_DT[x.dtype], _dev(codes, "codes"), _dev(scales, "scales"),
                                  M, N, K, block, _dev(y, "y"), _stream(stream)), "qwz_dequant_gemm")
    return y
