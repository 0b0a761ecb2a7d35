// zq_api.hip -- the C ABI declared in include/zq.h: argument validation on
// the host, grid sizing, and launches on the caller's stream.
//
// Every check runs before anything is enqueued, so an argument error writes
// no output byte.  The library allocates nothing; its only state is the
// static address table of the allocation-free gathered reduce.  Each
// launch covers its whole tensor (one tile per wave), so the grid size follows
// from n alone.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "zq.h"
#include "zq_host.h"
#include "zq_internal.h"

#ifndef ZQ_FIXED
#define ZQ_FIXED 1
#endif

namespace {

using namespace zq;

// Shared body of qwz_quantize / qgz_quantize.
int quantize(const void* x, int xt, int64_t n, int32_t block, uint8_t* out, float* scales, void* stream,
             int qbits) {
  if (n < 0) return ZQ_E_SIZE;
  const int lgB = log2_block(block);
  if (lgB < 0) return ZQ_E_BLOCK;
  if (!dtype_ok(xt)) return ZQ_E_DTYPE;
  if (n == 0) return ZQ_OK;
  if (!x || !out || !scales) return ZQ_E_NULL;
  if (!aligned(x, 16) || !aligned(out, 16) || !aligned(scales, 4)) return ZQ_E_ALIGN;
  const int64_t nb = num_scales(n, block);
  const int64_t out_bytes = qbits == 8 ? n : (n + 1) / 2;
  if (any_overlap({{out, out_bytes}, {scales, 4 * nb}}, {{x, n * elem_bytes(xt)}})) return ZQ_E_ALIAS;

  const int64_t nfull = n / block;
  const int64_t rest = n - nfull * block;
  const int64_t blocks_per_wave = 64 / (block / quant_elems((int)elem_bytes(xt), block));
  // workgroups of full blocks, plus one for a short last block
  const int64_t full_wgs =
      nfull > 0 ? grid_for((nfull + blocks_per_wave - 1) / blocks_per_wave,
                           kQuantThreads / 64 * quant_tiles((int)elem_bytes(xt)))
                : 0;
  if (nfull > 0 && full_wgs == 0) return ZQ_E_SIZE;
  const int64_t grid = full_wgs + (rest > 0 ? 1 : 0);
  if (grid > kMaxGrid) return ZQ_E_SIZE;

  return launch(quant_kernel(xt, qbits, lgB), (unsigned)grid, kQuantThreads, static_cast<hipStream_t>(stream), x,
                nfull, out, scales, (int)rest);
}

int dequantize(const void* codes, const float* scales, int64_t n, int32_t block, void* y, int yt, void* stream,
               int qbits) {
  if (n < 0) return ZQ_E_SIZE;
  const int lgB = log2_block(block);
  if (lgB < 0) return ZQ_E_BLOCK;
  if (!dtype_ok(yt)) return ZQ_E_DTYPE;
  if (n == 0) return ZQ_OK;
  if (!codes || !scales || !y) return ZQ_E_NULL;
  if (!aligned(codes, 16) || !aligned(y, 16) || !aligned(scales, 4)) return ZQ_E_ALIGN;
  const int64_t nb = num_scales(n, block);
  const int64_t in_bytes = qbits == 8 ? n : (n + 1) / 2;
  if (any_overlap({{y, n * elem_bytes(yt)}}, {{codes, in_bytes}, {scales, 4 * nb}})) return ZQ_E_ALIAS;

  // thread g < n/E dequantises elements [gE, gE + E); the n % E leftovers go
  // to the following threads, one element each
  const int64_t E = qbits == 8 ? deq8_elems((int)elem_bytes(yt)) : deq4_elems((int)elem_bytes(yt));
  const int64_t grid = grid_for(n / E + n % E, kDeqThreads);
  if (grid == 0) return ZQ_E_SIZE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  return launch(dequant_kernel(yt, qbits), (unsigned)grid, kDeqThreads, st, static_cast<const uint8_t*>(codes),
                scales, n, lgB, y);
}

// Shared body of qgz_reduce_level (fused = false: INT4 output only, both
// pointers required) and qgz_reduce_dequantize (fused = true: y of dtype yt
// required, the INT4 output optional -- both of its pointers or neither).
// Shared body of the reduce entry points.  gather: packed_in / scales_in are
// device tables of P slice pointers rather than the slices themselves.
int reduce(const uint8_t* packed_in, const float* scales_in, int32_t P, int64_t m, int32_t block,
           uint8_t* packed_out, float* scales_out, bool fused, void* y, int yt, void* stream, bool gather = false) {
  if (m < 0) return ZQ_E_SIZE;
  const int lgB = log2_block(block);
  if (lgB < 0) return ZQ_E_BLOCK;
  if (fused && !dtype_ok(yt)) return ZQ_E_DTYPE;
  if (P < 1 || P > 1024) return ZQ_E_P;
  if (m == 0) return ZQ_OK;
  if (!packed_in || !scales_in || (packed_out == nullptr) != (scales_out == nullptr)) return ZQ_E_NULL;
  if (fused ? y == nullptr : packed_out == nullptr) return ZQ_E_NULL;
  if (gather ? !aligned(packed_in, 8) || !aligned(scales_in, 8) : !aligned(packed_in, 16) || !aligned(scales_in, 4))
    return ZQ_E_ALIGN;
  if (packed_out && (!aligned(packed_out, 16) || !aligned(scales_out, 4))) return ZQ_E_ALIGN;
  if (fused && !aligned(y, 16)) return ZQ_E_ALIGN;
  const int64_t slice_bytes = (m + 1) / 2, nb = num_scales(m, block);
  // (gathered slices live elsewhere; only their pointer tables are checked)
  const Range ins[] = {{packed_in, gather ? 8 * (int64_t)P : slice_bytes * P},
                       {scales_in, gather ? 8 * (int64_t)P : 4 * nb * P}};
  Range outs[3];
  int nouts = 0;
  if (packed_out) {
    outs[nouts++] = {packed_out, slice_bytes};
    outs[nouts++] = {scales_out, 4 * nb};
  }
  if (fused) outs[nouts++] = {y, m * elem_bytes(yt)};
  for (int o = 0; o < nouts; ++o) {
    for (const Range& in : ins)
      if (overlap(outs[o], in)) return ZQ_E_ALIAS;
    for (int o2 = o + 1; o2 < nouts; ++o2)
      if (overlap(outs[o], outs[o2])) return ZQ_E_ALIAS;
  }

  // every slice starts 16-byte aligned when m % 32 == 0: vector path over
  // whole groups of blocks (4 wave tiles of 64 lanes x E elements each)
  const bool vector_path = m % 32 == 0;
  const int64_t full_blocks = vector_path ? m / block : 0;
  const int64_t waves_large = (full_blocks + 64 / (block / kReduceElems) - 1) / (64 / (block / kReduceElems));
  ReduceShape shape = ReduceShape::kLarge;
  if (block <= 512 && waves_large < ZQ_REDUCE_SMALL_WAVES) shape = ReduceShape::kSmall;
  else if (block <= 512 && P <= 2 && !fused) shape = ReduceShape::kTwoSlices;
  const int64_t group_blocks = kThreads / 64 * (64 / (block / reduce_elems(shape)));
  const int64_t groups = full_blocks / group_blocks;
  const int64_t nfull = groups * group_blocks;
  const int64_t grid = grid_for(groups, reduce_tiles(shape));
  if (grid == 0 && groups > 0) return ZQ_E_SIZE;

  // P = 2, 4, 8 on large levels: the kernel with the slice count fixed at
  // compile time (each workgroup takes reduce_fixed_tiles(P) groups)
  // and on small levels (one group per workgroup, the small-level group size)
  const bool small = shape == ReduceShape::kSmall;
  ReduceKernel fixed = !ZQ_FIXED ? nullptr
                       : small   ? reduce_fixed_small_kernel(lgB, P, fused ? yt : -1, gather)
                                 : reduce_fixed_kernel(lgB, P, fused ? yt : -1, gather);
  // (its groups: the same whole-group range [0, nfull) in its own group size)
  const int64_t fixed_groups =
      !fixed ? 0 : small ? groups : nfull / (kThreads / 64 * (64 / (block / reduce_fixed_elems())));
  const int64_t fixed_grid = !fixed ? 0 : small ? groups : grid_for(fixed_groups, reduce_fixed_tiles(P));
  if (fixed && fixed_grid == 0 && groups > 0) return ZQ_E_SIZE;

  hipStream_t st = static_cast<hipStream_t>(stream);
  if (groups > 0) {
    int rc = fixed ? launch(fixed, (unsigned)fixed_grid, kThreads, st, packed_in, scales_in, (int)P, slice_bytes, nb,
                            nfull, packed_out, scales_out, y)
                   : launch(gather ? reduce_gather_kernel(lgB, shape) : reduce_kernel(lgB, shape, fused ? yt : -1),
                            (unsigned)grid, kThreads, st, packed_in, scales_in, (int)P, slice_bytes, nb, nfull,
                            packed_out, scales_out, y);
    if (rc != ZQ_OK) return rc;
  }
  // remaining blocks (those after the last whole group, including a short
  // last block, or all of them when slices are not 16-byte aligned): one wave
  // per block
  for (int64_t b0 = nfull; b0 < nb; b0 += (1LL << 30)) {
    const int64_t cnt = (nb - b0) < (1LL << 30) ? (nb - b0) : (1LL << 30);
    int rc = launch(reduce_generic_kernel(gather), (unsigned)cnt, 64u, st, packed_in, scales_in, (int)P, slice_bytes,
                    nb, m,
                    (int)block, b0, packed_out, scales_out, fused ? y : nullptr, fused ? yt : 0);
    if (rc != ZQ_OK) return rc;
  }
  return ZQ_OK;
}

// Slice-address tables of qgz_reduce_level_gather_noalloc: one static array
// per GPU, held until the process ends (packed-slice addresses in entries
// [0, P), scale-slice addresses in [P, 2P)).  Host code never uses this name
// as an address: the device address comes from hipGetSymbolAddress, once per
// device (scratch_on_current_device).
constexpr int kScratchEntries = 2 * 1024;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) uint64_t scratch[kScratchEntries];

// Device address of `scratch` on the current device (looked up on the
// first call on each device, with that device current); ZQ_E_HIP if HIP
// cannot give it.
int scratch_on_current_device(uint64_t** out) {
  static std::once_flag once[kMaxDevices];
  static uint64_t* addr[kMaxDevices];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return ZQ_E_HIP;
  std::call_once(once[dev], [dev] {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess) addr[dev] = static_cast<uint64_t*>(p);
  });
  if (addr[dev] == nullptr) return ZQ_E_HIP;
  *out = addr[dev];
  return ZQ_OK;
}

// The reduce level over slices whose addresses are in host arrays: the
// addresses are checked on the host, written into this device's scratch
// table by fill kernels on the stream (their values travel as kernel
// arguments), and the gathered reduce reads them from there.
int reduce_gather_host(const uint8_t* const* packed_slices, const float* const* scale_slices, int32_t P, int64_t m,
                       int32_t block, uint8_t* packed_out, float* scales_out, void* stream) {
  if (m < 0) return ZQ_E_SIZE;
  if (log2_block(block) < 0) return ZQ_E_BLOCK;
  if (P < 1 || 2 * (int64_t)P > kScratchEntries) return ZQ_E_P;
  if (m == 0) return ZQ_OK;
  if (!packed_slices || !scale_slices || !packed_out || !scales_out) return ZQ_E_NULL;
  const int64_t slice_bytes = (m + 1) / 2, nb = num_scales(m, block);
  const Range outs[] = {{packed_out, slice_bytes}, {scales_out, 4 * nb}};
  for (int32_t p = 0; p < P; ++p) {
    if (!packed_slices[p] || !scale_slices[p]) return ZQ_E_NULL;
    if ((m % 32 == 0 && !aligned(packed_slices[p], 16)) || !aligned(scale_slices[p], 4)) return ZQ_E_ALIGN;
    const Range ins[] = {{packed_slices[p], slice_bytes}, {scale_slices[p], 4 * nb}};
    for (const Range& o : outs)
      for (const Range& i : ins)
        if (overlap(o, i)) return ZQ_E_ALIAS;
  }
  uint64_t* table = nullptr;
  int rc = scratch_on_current_device(&table);
  if (rc != ZQ_OK) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t entries = 2 * (int64_t)P;
  for (int64_t e0 = 0; e0 < entries; e0 += kTableChunk) {
    TableChunk chunk;
    const int count = (int)(entries - e0 < kTableChunk ? entries - e0 : kTableChunk);
    for (int k = 0; k < count; ++k) {
      const int64_t e = e0 + k;
      chunk.v[k] = e < P ? reinterpret_cast<uint64_t>(packed_slices[e]) : reinterpret_cast<uint64_t>(scale_slices[e - P]);
    }
    for (int k = count; k < kTableChunk; ++k) chunk.v[k] = 0;
    rc = launch(fill_table_kernel(), 1u, (unsigned)kTableChunk, st, table + e0, chunk, count);
    if (rc != ZQ_OK) return rc;
  }
  return reduce(reinterpret_cast<const uint8_t*>(table), reinterpret_cast<const float*>(table + P), P, m, block,
                packed_out, scales_out, false, nullptr, -1, stream, true);
}

}  // namespace

extern "C" {

int qwz_quantize(const void* x, zq_dtype xt, int64_t n, int32_t block, int8_t* codes, float* scales,
                 void* stream) {
  return quantize(x, xt, n, block, reinterpret_cast<uint8_t*>(codes), scales, stream, 8);
}

int qwz_dequantize(const int8_t* codes, const float* scales, int64_t n, int32_t block, void* y, zq_dtype yt,
                   void* stream) {
  return dequantize(codes, scales, n, block, y, yt, stream, 8);
}

int qgz_quantize(const void* g, zq_dtype gt, int64_t n, int32_t block, uint8_t* packed, float* scales,
                 void* stream) {
  return quantize(g, gt, n, block, packed, scales, stream, 4);
}

int qgz_dequantize(const uint8_t* packed, const float* scales, int64_t n, int32_t block, void* y, zq_dtype yt,
                   void* stream) {
  return dequantize(packed, scales, n, block, y, yt, stream, 4);
}

int qgz_reduce_level(const uint8_t* packed_in, const float* scales_in, int32_t P, int64_t m, int32_t block,
                     uint8_t* packed_out, float* scales_out, void* stream) {
  return reduce(packed_in, scales_in, P, m, block, packed_out, scales_out, false, nullptr, -1, stream);
}

int qgz_reduce_dequantize(const uint8_t* packed_in, const float* scales_in, int32_t P, int64_t m, int32_t block,
                          void* y, zq_dtype yt, uint8_t* packed_out, float* scales_out, void* stream) {
  return reduce(packed_in, scales_in, P, m, block, packed_out, scales_out, true, y, yt, stream);
}

int qgz_reduce_level_gather(const uint8_t* const* packed_slices, const float* const* scale_slices, int32_t P,
                            int64_t m, int32_t block, uint8_t* packed_out, float* scales_out, void* stream) {
  return reduce(reinterpret_cast<const uint8_t*>(packed_slices), reinterpret_cast<const float*>(scale_slices), P, m,
                block, packed_out, scales_out, false, nullptr, -1, stream, true);
}

int qgz_reduce_level_gather_noalloc(const uint8_t* const* packed_slices, const float* const* scale_slices, int32_t P,
                                    int64_t m, int32_t block, uint8_t* packed_out, float* scales_out, void* stream) {
  return reduce_gather_host(packed_slices, scale_slices, P, m, block, packed_out, scales_out, stream);
}

int64_t zq_num_scales(int64_t n, int32_t block) {
  if (n < 0 || log2_block(block) < 0) return -1;
  return num_scales(n, block);
}

int64_t zq_int4_bytes(int64_t n) { return n < 0 ? -1 : (n + 1) / 2; }

const char* zq_status_string(int status) {
  switch (status) {
    case ZQ_OK: return "ok";
    case ZQ_E_NULL: return "null pointer";
    case ZQ_E_BLOCK: return "block must be a power of two in [32, 1024]";
    case ZQ_E_DTYPE: return "unknown dtype";
    case ZQ_E_ALIGN: return "misaligned pointer (elements/codes 16 B, scales 4 B)";
    case ZQ_E_SIZE: return "negative size";
    case ZQ_E_P: return "slice count outside [1, 1024]";
    case ZQ_E_HIP: return "HIP launch failed";
    case ZQ_E_ALIAS: return "an output overlaps an input";
    default: return "unknown status";
  }
}

}  // extern "C"
