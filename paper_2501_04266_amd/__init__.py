"""MI355X-native qwZ / qgZ compression path (block-wise INT8 weight and INT4
gradient quantisation with a multi-slice dequant-sum-requant reduction), as
used by the hierarchical ZeRO++ partitioning of arXiv 2501.04266.

The compute runs in the HIP library libzq.so (C ABI in include/zq.h); this
package is its Python binding.  Importing it does not need a GPU; calling a
kernel does.
"""
from ._lib import (  # noqa: F401
    LIB_PATH,
    STATUS,
    ZQError,
    gather_tables,
    int4_bytes,
    lib,
    num_scales,
    qgz_dequantize,
    qgz_quantize,
    qgz_reduce_dequantize,
    qgz_reduce_level,
    qgz_reduce_level_gather,
    qgz_reduce_level_gather_noalloc,
    qwz_dequant_gemm,
    qwz_dequantize,
    qwz_quantize,
)
