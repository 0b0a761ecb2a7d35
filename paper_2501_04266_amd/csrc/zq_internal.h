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

// Workgroups are dealt round-robin to the 8 XCDs (each with its own L2).
// With the remap on, a launch is rounded up to a multiple of 8 workgroups
// and workgroup i takes tile (i % 8) * (grid / 8) + i / 8, so every XCD
// streams one contiguous range and neighbouring tiles share an L2.  It pays
// for the INT8 dequantiser, whose 16 lanes per block all read the block's
// scale (one L2 instead of several fetching each scale line); the read-heavy
// kernels measured slower with it, so they keep the round-robin order.
#ifndef ZQ_REMAP_DEQ8
#define ZQ_REMAP_DEQ8 1
#endif
constexpr int kXcds = 8;
inline int64_t launch_grid(int64_t tiles, bool remap) {
  return remap ? (tiles + kXcds - 1) / kXcds * kXcds : tiles;
}

// Elements per lane.  Each wave handles one tile of 64 lanes x E elements and
// each workgroup four tiles; launches cover the whole tensor (no grid-stride
// loop), which measured fastest for streaming on gfx950.  Loads stay at 16 B
// per lane where possible and each lane writes at most 32 contiguous bytes
// (wider per-lane writes lose bandwidth).
#ifndef ZQ_QUANT_E_F32
#define ZQ_QUANT_E_F32 4
#endif
#ifndef ZQ_QUANT_E_16
#define ZQ_QUANT_E_16 8
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
#define ZQ_DEQ4_E_F32 8
#endif
#ifndef ZQ_DEQ4_E_16
#define ZQ_DEQ4_E_16 16
#endif
constexpr int deq8_elems(int out_bytes) { return out_bytes == 4 ? ZQ_DEQ8_E_F32 : ZQ_DEQ8_E_16; }
constexpr int deq4_elems(int out_bytes) { return out_bytes == 4 ? ZQ_DEQ4_E_F32 : ZQ_DEQ4_E_16; }
constexpr int kReduceElems = 32;  // 16 bytes of every slice per lane

using QuantKernel = void (*)(const void*, int64_t, uint8_t*, float*);
using QuantTailKernel = void (*)(const void*, int64_t, int, uint8_t*, float*);
using Dequant8Kernel = void (*)(const int8_t*, const float*, int64_t, int, void*);
using Dequant4Kernel = void (*)(const uint8_t*, const float*, int64_t, int, void*);
using ReduceKernel = void (*)(const uint8_t*, const float*, int, int64_t, int64_t, int64_t, uint8_t*, float*);
using ReduceGenericKernel = void (*)(const uint8_t*, const float*, int, int64_t, int64_t, int64_t, int, int64_t,
                                     uint8_t*, float*);

QuantKernel quant_kernel(int dt, int qbits, int lgB);
QuantTailKernel quant_tail_kernel(int dt, int qbits);
Dequant8Kernel dequant8_kernel(int dt);
Dequant4Kernel dequant4_kernel(int dt);
ReduceKernel reduce_kernel(int lgB);
ReduceGenericKernel reduce_generic_kernel();

}  // namespace zq
