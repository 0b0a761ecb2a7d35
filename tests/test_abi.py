"""CPU tests of the C ABI boundary (no kernel is launched).

The library must load and export every function include/zq.h declares; the
host-only helpers and every argument check (which runs before anything is
enqueued) are exercised with fake device pointers.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "zq.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w\s\*]*?\b([a-z_][a-z0-9_]*)\s*\(", src, re.M)))


@pytest.fixture(scope="module")
def L():
    from paper_2501_04266_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2501_04266_amd import build
        build.build()
    return _lib.lib()


def test_header_declares_the_five_calls():
    names = _declared()
    for fn in ("qwz_quantize", "qwz_dequantize", "qgz_quantize", "qgz_reduce_level", "qgz_dequantize",
               "qgz_reduce_dequantize", "qgz_reduce_level_gather", "qwz_dequant_gemm", "zq_num_scales",
               "zq_int4_bytes", "zq_status_string"):
        assert fn in names, fn


def test_every_declared_symbol_is_exported(L):
    for fn in _declared():
        assert hasattr(L, fn), f"libzq.so does not export {fn}"


def test_binding_names_match_header():
    from paper_2501_04266_amd import _lib
    assert sorted(_lib.EXPORTS) == _declared()


def test_size_helpers(L):
    assert L.zq_num_scales(0, 256) == 0
    assert L.zq_num_scales(1, 256) == 1
    assert L.zq_num_scales(123_456_789, 256) == 482_254
    assert L.zq_num_scales(123_456_789, 64) == 1_929_013
    assert L.zq_num_scales(10, 48) == -1
    assert L.zq_num_scales(-1, 64) == -1
    assert L.zq_int4_bytes(123_456_789) == 61_728_395
    assert L.zq_int4_bytes(-3) == -1
    for st in range(-8, 1):
        assert L.zq_status_string(st)
    assert L.zq_status_string(-99) == b"unknown status"


# fake, suitably aligned "device" addresses: validation never dereferences them
A = 0x7F0000000000
B = 0x7F0010000000
C = 0x7F0020000000


@pytest.mark.parametrize("call,args,status", [
    ("qwz_quantize", (A, 0, -1, 256, B, C, None), -5),
    ("qwz_quantize", (A, 0, 100, 48, B, C, None), -2),
    ("qwz_quantize", (A, 0, 100, 16, B, C, None), -2),
    ("qwz_quantize", (A, 0, 100, 2048, B, C, None), -2),
    ("qwz_quantize", (A, 7, 100, 256, B, C, None), -3),
    ("qwz_quantize", (None, 0, 100, 256, B, C, None), -1),
    ("qwz_quantize", (A, 0, 100, 256, None, C, None), -1),
    ("qwz_quantize", (A + 4, 0, 100, 256, B, C, None), -4),
    ("qwz_quantize", (A, 0, 100, 256, B + 8, C, None), -4),
    ("qwz_quantize", (A, 0, 100, 256, B, C + 2, None), -4),
    ("qwz_quantize", (A, 0, 100, 256, A + 256, C, None), -8),
    ("qwz_quantize", (A, 0, 100, 256, B, A + 396, None), -8),
    ("qwz_quantize", (A, 0, 0, 256, None, None, None), 0),
    ("qwz_dequantize", (A, C, 100, 256, A + 96, 2, None), -8),
    ("qwz_dequantize", (A, C, 100, 256, B, 3, None), -3),
    ("qwz_dequantize", (A, None, 100, 256, B, 2, None), -1),
    ("qwz_dequantize", (A, C, 0, 256, B, 2, None), 0),
    # packed output of 100 elements is 50 bytes: scales at +48 overlap it
    ("qgz_quantize", (A, 0, 100, 64, B, B + 48, None), -8),
    # bf16 input of 1001 elements spans 2002 bytes: output at +2000 overlaps it
    ("qgz_quantize", (A, 2, 1001, 64, A + 2000, C, None), -8),
    ("qgz_dequantize", (A, C, 1001, 64, B + 4, 0, None), -4),
])
def test_argument_errors(L, call, args, status):
    conv = [ctypes.c_void_p(a) if isinstance(a, int) and a > 1 << 20 else a for a in args]
    got = getattr(L, call)(*conv)
    assert got == status, f"{call}{args}: got {got}, want {status}"


def test_reduce_argument_errors(L):
    f = L.qgz_reduce_level
    vp = ctypes.c_void_p
    assert f(vp(A), vp(C), 0, 256, 128, vp(B), vp(B + 4096), None) == -6
    assert f(vp(A), vp(C), 1025, 256, 128, vp(B), vp(B + 4096), None) == -6
    assert f(vp(A), vp(C), 8, -1, 128, vp(B), vp(B + 4096), None) == -5
    assert f(vp(A), vp(C), 8, 256, 100, vp(B), vp(B + 4096), None) == -2
    assert f(vp(A), vp(C), 8, 0, 128, None, None, None) == 0
    assert f(vp(A), None, 8, 256, 128, vp(B), vp(B + 4096), None) == -1
    assert f(vp(A + 8), vp(C), 8, 256, 128, vp(B), vp(B + 4096), None) == -4
    # output overlapping slice 3 of the input
    assert f(vp(A), vp(C), 8, 256, 128, vp(A + 3 * 128), vp(B + 4096), None) == -8
    # output scales overlapping input scales
    assert f(vp(A), vp(C), 8, 256, 128, vp(B), vp(C + 8), None) == -8


def test_reduce_dequantize_argument_errors(L):
    f = L.qgz_reduce_dequantize
    vp = ctypes.c_void_p
    Y = 0x7F0030000000
    assert f(vp(A), vp(C), 8, 256, 128, vp(Y), 5, None, None, None) == -3      # bad dtype
    assert f(vp(A), vp(C), 8, 256, 128, vp(Y), -1, None, None, None) == -3     # bad dtype, no INT4 output
    assert f(vp(A), vp(C), 0, 256, 128, vp(Y), 0, None, None, None) == -6
    assert f(vp(A), vp(C), 8, 256, 96, vp(Y), 0, None, None, None) == -2
    assert f(vp(A), vp(C), 8, -4, 128, vp(Y), 0, None, None, None) == -5
    assert f(vp(A), vp(C), 8, 0, 128, None, 0, None, None, None) == 0
    assert f(vp(A), vp(C), 8, 256, 128, None, 0, None, None, None) == -1       # y required
    assert f(vp(A), vp(C), 8, 256, 128, vp(Y), 0, vp(B), None, None) == -1     # one INT4 pointer only
    assert f(vp(A), vp(C), 8, 256, 128, vp(Y + 4), 0, None, None, None) == -4
    assert f(vp(A), vp(C), 8, 256, 128, vp(A + 512), 0, None, None, None) == -8  # y over the slices
    assert f(vp(A), vp(C), 8, 256, 128, vp(Y), 0, vp(Y + 512), vp(B), None) == -8  # y over packed_out
    # the plain reduce still requires its INT4 outputs
    assert L.qgz_reduce_level(vp(A), vp(C), 8, 256, 128, None, None, None) == -1


def test_dequant_gemm_argument_errors(L):
    f = L.qwz_dequant_gemm
    vp = ctypes.c_void_p
    Y = 0x7F0030000000
    # (x, xt, codes, scales, M, N, K, block, y)
    assert f(vp(A), 0, vp(B), vp(C), 4, 4, 64, 256, vp(Y), None) == -3      # fp32 x not supported
    assert f(vp(A), 2, vp(B), vp(C), 4, 4, 96, 256, vp(Y), None) == -5      # K not a multiple of 64
    assert f(vp(A), 2, vp(B), vp(C), -1, 4, 64, 256, vp(Y), None) == -5
    assert f(vp(A), 2, vp(B), vp(C), 4, 4, 64, 100, vp(Y), None) == -2
    assert f(vp(A), 2, vp(B), vp(C), 0, 4, 64, 256, None, None) == 0        # empty output: no-op
    assert f(vp(A), 2, vp(B), vp(C), 4, 4, 64, 256, None, None) == -1
    assert f(None, 2, vp(B), vp(C), 4, 4, 64, 256, vp(Y), None) == -1
    assert f(vp(A + 8), 2, vp(B), vp(C), 4, 4, 64, 256, vp(Y), None) == -4
    assert f(vp(A), 2, vp(B + 4), vp(C), 4, 4, 64, 256, vp(Y), None) == -4
    assert f(vp(A), 1, vp(B), vp(C), 4, 4, 64, 256, vp(Y + 2), None) == -4
    # y (4 x 4 floats) over the end of x (4 x 64 bf16 = 512 bytes)
    assert f(vp(A), 2, vp(B), vp(C), 4, 4, 64, 256, vp(A + 500), None) == -8
    # y over the scales
    assert f(vp(A), 2, vp(B), vp(C), 4, 4, 64, 256, vp(C), None) == -8


def test_binding_rejects_undersized_or_mistyped_buffers():
    """The C ABI takes raw pointers; the binding checks every buffer's size and
    dtype on the host before anything reaches the library (CPU tensors are
    enough: these checks come first)."""
    import torch

    import paper_2501_04266_amd as zq
    x = torch.zeros(1000)
    with pytest.raises(ValueError):
        zq.qwz_quantize(x, 256, codes=torch.zeros(999, dtype=torch.int8), scales=torch.zeros(4))
    with pytest.raises(ValueError):
        zq.qwz_quantize(x, 256, codes=torch.zeros(1000, dtype=torch.int8), scales=torch.zeros(3))
    with pytest.raises(TypeError):
        zq.qwz_quantize(x, 256, codes=torch.zeros(1000, dtype=torch.int16), scales=torch.zeros(4))
    with pytest.raises(TypeError):
        zq.qwz_quantize(torch.zeros(1000, dtype=torch.int32), 256)
    with pytest.raises(ValueError):
        zq.qgz_quantize(x, 128, packed=torch.zeros(499, dtype=torch.uint8), scales=torch.zeros(8))
    with pytest.raises(ValueError):
        zq.qgz_dequantize(torch.zeros(500, dtype=torch.uint8), torch.zeros(8), 1000, 128, y=torch.zeros(999))
    with pytest.raises(ValueError):
        zq.qgz_reduce_level(torch.zeros(999, dtype=torch.uint8), torch.zeros(16), 2, 1000, 128)
    with pytest.raises(ValueError):
        zq.qgz_reduce_level(torch.zeros(1000, dtype=torch.uint8), torch.zeros(16), 2, 1000, 128,
                            packed_out=torch.zeros(10, dtype=torch.uint8), scales_out=torch.zeros(8))
    with pytest.raises(ValueError):
        zq.qgz_reduce_dequantize(torch.zeros(1000, dtype=torch.uint8), torch.zeros(16), 2, 1000, 128,
                                 y=torch.zeros(999))
    with pytest.raises(ValueError):
        zq.qwz_dequant_gemm(torch.zeros((4, 64), dtype=torch.bfloat16), torch.zeros(8 * 64, dtype=torch.int8),
                            torch.zeros(2), 8, 256, y=torch.zeros((4, 7)))
    with pytest.raises(TypeError):
        zq.qwz_dequant_gemm(torch.zeros((4, 64)), torch.zeros(8 * 64, dtype=torch.int8), torch.zeros(2), 8, 256)


def test_reduce_gather_argument_errors(L):
    f = L.qgz_reduce_level_gather
    vp = ctypes.c_void_p
    T, S = 0x7F0040000000, 0x7F0040001000       # device pointer tables (8-byte aligned)
    assert f(vp(T), vp(S), 0, 256, 128, vp(B), vp(B + 4096), None) == -6
    assert f(vp(T), vp(S), 8, 256, 100, vp(B), vp(B + 4096), None) == -2
    assert f(vp(T), vp(S), 8, -1, 128, vp(B), vp(B + 4096), None) == -5
    assert f(None, vp(S), 8, 256, 128, vp(B), vp(B + 4096), None) == -1
    assert f(vp(T + 4), vp(S), 8, 256, 128, vp(B), vp(B + 4096), None) == -4   # table not 8-byte aligned
    assert f(vp(T), vp(S), 8, 256, 128, vp(T + 32), vp(B + 4096), None) == -8  # output over the table
    assert f(vp(T), vp(S), 8, 0, 128, None, None, None) == 0


def test_reduce_gather_noalloc_argument_errors(L):
    """Every check of the allocation-free gathered reduce runs on the host
    arrays of slice addresses before anything is enqueued."""
    f = L.qgz_reduce_level_gather_noalloc
    vp = ctypes.c_void_p
    P, m, block = 4, 4096, 128
    base = 0x7F0050000000

    def tabs(packed, scales):
        return (ctypes.c_void_p * len(packed))(*packed), (ctypes.c_void_p * len(scales))(*scales)

    pk = [base + p * 0x10000 for p in range(P)]
    sc = [base + 0x100000 + p * 0x1000 for p in range(P)]
    out, sout = base + 0x200000, base + 0x300000
    tp, ts = tabs(pk, sc)
    assert f(tp, ts, 0, m, block, vp(out), vp(sout), None) == -6
    assert f(tp, ts, 1025, m, block, vp(out), vp(sout), None) == -6          # beyond the 1024-pair table
    assert f(tp, ts, P, m, 100, vp(out), vp(sout), None) == -2
    assert f(tp, ts, P, -1, block, vp(out), vp(sout), None) == -5
    assert f(None, ts, P, m, block, vp(out), vp(sout), None) == -1
    assert f(tp, ts, P, m, block, None, vp(sout), None) == -1
    tq, tt = tabs(pk[:2] + [0] + pk[3:], sc)
    assert f(tq, tt, P, m, block, vp(out), vp(sout), None) == -1             # a null slice
    tq, tt = tabs(pk[:2] + [pk[2] + 8] + pk[3:], sc)
    assert f(tq, tt, P, m, block, vp(out), vp(sout), None) == -4             # slice not 16-byte aligned (m % 32 == 0)
    tq, tt = tabs(pk, sc[:1] + [sc[1] + 2] + sc[2:])
    assert f(tq, tt, P, m, block, vp(out), vp(sout), None) == -4             # scale slice not 4-byte aligned
    assert f(tp, ts, P, m, block, vp(pk[3] + 16), vp(sout), None) == -8     # output over a slice
    assert f(tp, ts, P, m, block, vp(out), vp(sc[0]), None) == -8           # scales over a scale slice
    assert f(tp, ts, P, 0, block, None, None, None) == 0
