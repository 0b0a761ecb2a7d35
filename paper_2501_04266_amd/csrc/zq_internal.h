// zq_internal.h -- launch geometry and kernel handles shared by the kernel and
// API translation units.
#pragma once
#include <stdint.h>

namespace zq {

constexpr int kThreads = 256;  // threads per workgroup of the streaming kernels (4 waves)
#ifndef ZQ_QUANT_THREADS
#define ZQ_QUANT_THREADS 256
#endif
constexpr int kQuantThreads = ZQ_QUANT_THREADS;
// wave tiles per wave in the quantiser: one for either input width (two
// tiles on 16-bit input measured slower than one tile of 16 elements per
// lane; on fp32 input two tiles measured slower too)
#ifndef ZQ_QUANT_TILES_F32
#define ZQ_QUANT_TILES_F32 1
#endif
#ifndef ZQ_QUANT_TILES_16
#define ZQ_QUANT_TILES_16 1
#endif
constexpr int quant_tiles(int dt_bytes) { return dt_bytes == 4 ? ZQ_QUANT_TILES_F32 : ZQ_QUANT_TILES_16; }
#ifndef ZQ_DEQ_THREADS
#define ZQ_DEQ_THREADS 256
#endif
constexpr int kDeqThreads = ZQ_DEQ_THREADS;


// Elements per lane.  Each wave handles one tile of 64 lanes x E elements and
// each workgroup four tiles; launches cover the whole tensor (no grid-stride
// loop), which measured fastest for streaming on gfx950.  Loads are 16 B per
// lane and instruction (a quantiser lane holding more takes several 16-byte
// chunks of its block, so each load instruction stays contiguous across the
// block's lanes) and each lane writes at most 32 contiguous bytes (wider
// per-lane writes lose bandwidth).  Quantiser: 4 elements per lane on fp32
// input (8 or 16, with half or a quarter of the VALU instructions per
// element, measured 3-5% slower), 16 on 16-bit input (2-3% faster than 8).
#ifndef ZQ_QUANT_E_F32
#define ZQ_QUANT_E_F32 4
#endif
#ifndef ZQ_QUANT_E_16
#define ZQ_QUANT_E_16 16
#endif
constexpr int quant_elems(int dt_bytes, int block) {
  int e = dt_bytes == 4 ? ZQ_QUANT_E_F32 : ZQ_QUANT_E_16;
  return block / e > 64 ? block / 64 : e;  // a block may span at most one wave
}
#ifndef ZQ_DEQ8_E_F32
#define ZQ_DEQ8_E_F32 8
#endif
#ifndef ZQ_DEQ8_E_16
#define ZQ_DEQ8_E_16 8
#endif
#ifndef ZQ_DEQ4_E_F32
#define ZQ_DEQ4_E_F32 16
#endif
#ifndef ZQ_DEQ4_E_16
#define ZQ_DEQ4_E_16 16
#endif
constexpr int deq8_elems(int out_bytes) { return out_bytes == 4 ? ZQ_DEQ8_E_F32 : ZQ_DEQ8_E_16; }
constexpr int deq4_elems(int out_bytes) { return out_bytes == 4 ? ZQ_DEQ4_E_F32 : ZQ_DEQ4_E_16; }
#ifndef ZQ_REDUCE_E
#define ZQ_REDUCE_E 32
#endif
constexpr int kReduceElems = ZQ_REDUCE_E;  // 16 bytes of every slice per lane
constexpr int kReduceElemsSmall = 8;  // 4 bytes per slice per lane, for small levels
// Launch shapes of the reduce level (see the kernel): 32 elements per lane
// and 4-slice batches; the same with 2-slice batches for P <= 2; 8 elements
// per lane and 16-slice batches for levels with few waves.  TR = groups of 4
// wave tiles per workgroup, processed as one pipelined sequence.
#ifndef ZQ_REDUCE_TR
#define ZQ_REDUCE_TR 1
#endif
#ifndef ZQ_REDUCE_TR2
#define ZQ_REDUCE_TR2 2
#endif
#ifndef ZQ_REDUCE_TR_SMALL
#define ZQ_REDUCE_TR_SMALL 1
#endif
enum class ReduceShape { kLarge, kTwoSlices, kSmall };
constexpr int reduce_elems(ReduceShape s) { return s == ReduceShape::kSmall ? kReduceElemsSmall : kReduceElems; }
constexpr int reduce_tiles(ReduceShape s) {
  return s == ReduceShape::kTwoSlices ? ZQ_REDUCE_TR2 : s == ReduceShape::kSmall ? ZQ_REDUCE_TR_SMALL : ZQ_REDUCE_TR;
}
// A level whose E = 32 launch would have fewer waves than this runs the small
// variant (4x the waves, more slices in flight per wave).
#ifndef ZQ_REDUCE_SMALL_WAVES
#define ZQ_REDUCE_SMALL_WAVES 4096
#endif

// (x, full blocks, out, scales, length of the short last block or 0)
using QuantKernel = void (*)(const void*, int64_t, uint8_t*, float*, int);
using DequantKernel = void (*)(const uint8_t*, const float*, int64_t, int, void*);
using ReduceKernel = void (*)(const uint8_t*, const float*, int, int64_t, int64_t, int64_t, uint8_t*, float*, void*);
using ReduceGenericKernel = void (*)(const uint8_t*, const float*, int, int64_t, int64_t, int64_t, int, int64_t,
                                     uint8_t*, float*, void*, int);

QuantKernel quant_kernel(int dt, int qbits, int lgB);
DequantKernel dequant_kernel(int dt, int qbits);
// ydt < 0: INT4 output only; otherwise also the fused dequantisation to ydt
ReduceKernel reduce_kernel(int lgB, ReduceShape shape, int ydt);
// slices through device tables of P pointers (bytes, scales); INT4 output only
ReduceKernel reduce_gather_kernel(int lgB, ReduceShape shape);
ReduceGenericKernel reduce_generic_kernel(bool gather);
// vector-path kernel with the slice count fixed at compile time, for P = 2, 4
// or 8 and B = 64, 128 or 256 (ydt < 0: INT4 output only; gather: slices
// through pointer tables, INT4 output only); null where there is none.  Each
// workgroup takes reduce_fixed_tiles(P) groups.
ReduceKernel reduce_fixed_kernel(int lgB, int P, int ydt, bool gather);
// The same for small levels (the small-level lane width, one group per
// workgroup), P = 2, 4, 8; null otherwise.
ReduceKernel reduce_fixed_small_kernel(int lgB, int P, int ydt, bool gather);
// a chunk of 64-bit table entries passed by value to the table-fill kernel
constexpr int kTableChunk = 64;
struct TableChunk {
  uint64_t v[kTableChunk];
};
using FillTableKernel = void (*)(uint64_t*, TableChunk, int);
FillTableKernel fill_table_kernel();
int reduce_fixed_tiles(int P);
int reduce_fixed_elems();  // elements per lane of that kernel

}  // namespace zq
