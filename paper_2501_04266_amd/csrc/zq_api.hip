// zq_api.hip -- the C ABI declared in include/zq.h: argument validation on
// the host, grid sizing, and launches on the caller's stream.
//
// Every check runs before anything is enqueued, so an argument error writes
// no output byte.  The library allocates nothing and keeps no state.  Each
// launch covers its whole tensor (one tile per wave), so the grid size follows
// from n alone.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <tuple>
#include <utility>

#include "zq.h"
#include "zq_internal.h"

namespace {

using namespace zq;

constexpr int64_t kMaxGrid = 0x7fffffff;  // workgroups per launch

// Workgroups to cover `units` at `units_per_wg` each (0 if it exceeds the
// launch limit; callers turn that into ZQ_E_SIZE before anything is enqueued).
int64_t grid_for(int64_t units, int64_t units_per_wg) {
  int64_t g = (units + units_per_wg - 1) / units_per_wg;
  if (g < 1) g = 1;
  return g > kMaxGrid ? 0 : g;
}

// Launch with the kernel's exact parameter types; returns ZQ_E_HIP when the
// runtime rejects the launch.
template <typename... KArgs, typename... Args>
int launch(void (*kern)(KArgs...), unsigned grid, unsigned block, hipStream_t st, Args&&... args) {
  std::tuple<KArgs...> tup(std::forward<Args>(args)...);
  void* argv[sizeof...(KArgs)];
  std::apply([&](auto&... a) {
    int i = 0;
    ((argv[i++] = static_cast<void*>(&a)), ...);
  }, tup);
  hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(kern), dim3(grid), dim3(block), argv, 0, st);
  return e == hipSuccess ? ZQ_OK : ZQ_E_HIP;
}

int log2_block(int32_t block) {
  if (block < 32 || block > 1024 || (block & (block - 1)) != 0) return -1;
  int lg = 0;
  while ((1 << lg) < block) ++lg;
  return lg;
}

bool dtype_ok(int dt) { return dt == ZQ_F32 || dt == ZQ_F16 || dt == ZQ_BF16; }
int64_t elem_bytes(int dt) { return dt == ZQ_F32 ? 4 : 2; }
bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

struct Range {
  const void* p;
  int64_t bytes;
};
bool overlap(Range a, Range b) {
  uintptr_t a0 = reinterpret_cast<uintptr_t>(a.p), b0 = reinterpret_cast<uintptr_t>(b.p);
  return a0 < b0 + (uintptr_t)b.bytes && b0 < a0 + (uintptr_t)a.bytes;
}
bool any_overlap(std::initializer_list<Range> outs, std::initializer_list<Range> ins) {
  for (const Range& o : outs) {
    for (const Range& i : ins)
      if (overlap(o, i)) return true;
  }
  // outputs must not overlap each other either
  for (auto o1 = outs.begin(); o1 != outs.end(); ++o1)
    for (auto o2 = o1 + 1; o2 != outs.end(); ++o2)
      if (overlap(*o1, *o2)) return true;
  return false;
}

int64_t num_scales(int64_t n, int32_t block) { return (n + block - 1) / block; }

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
  const int64_t blocks_per_wave = 64 / (block / quant_elems((int)elem_bytes(xt), block));
  const int64_t grid = grid_for((nfull + blocks_per_wave - 1) / blocks_per_wave, kQuantThreads / 64 * kQuantTiles);
  if (grid == 0) return ZQ_E_SIZE;

  hipStream_t st = static_cast<hipStream_t>(stream);
  int rc = ZQ_OK;
  if (nfull > 0) {
    rc = launch(quant_kernel(xt, qbits, lgB), (unsigned)grid, kQuantThreads, st, x, nfull, out, scales);
    if (rc != ZQ_OK) return rc;
  }
  const int64_t rest = n - nfull * block;
  if (rest > 0) {
    rc = launch(quant_tail_kernel(xt, qbits), 1u, 64u, st, x, nfull * (int64_t)block, (int)rest, out,
                scales + nfull);
  }
  return rc;
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

  hipStream_t st = static_cast<hipStream_t>(stream);
  if (groups > 0) {
    int rc = launch(gather ? reduce_gather_kernel(lgB, shape) : reduce_kernel(lgB, shape, fused ? yt : -1),
                    (unsigned)grid, kThreads, st, packed_in, scales_in, (int)P, slice_bytes, nb, nfull, packed_out,
                    scales_out, y);
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

int qwz_dequant_gemm(const void* x, zq_dtype xt, const int8_t* codes, const float* scales, int64_t M, int64_t N,
                     int64_t K, int32_t block, float* y, void* stream) {
  if (M < 0 || N < 0 || K < 0) return ZQ_E_SIZE;
  const int lgB = log2_block(block);
  if (lgB < 0) return ZQ_E_BLOCK;
  if (xt != ZQ_BF16 && xt != ZQ_F16) return ZQ_E_DTYPE;
  if (K % kDqGemmK != 0) return ZQ_E_SIZE;
  if (M == 0 || N == 0) return ZQ_OK;
  if (!y || (K > 0 && (!x || !codes || !scales))) return ZQ_E_NULL;
  if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(scales, 4) || !aligned(y, 4)) return ZQ_E_ALIGN;
  if (any_overlap({{y, 4 * M * N}}, {{x, 2 * M * K}, {codes, N * K}, {scales, 4 * num_scales(N * K, block)}}))
    return ZQ_E_ALIAS;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const uint16_t* xh = static_cast<const uint16_t*>(x);
  if (M > ZQ_GEMM_SMALL_M) {
    const int64_t mtiles = (M + kDqGemmTileM - 1) / kDqGemmTileM, ntiles = (N + kDqGemmTileN - 1) / kDqGemmTileN;
    if (mtiles * ntiles > kMaxGrid) return ZQ_E_SIZE;
    return launch(dqgemm_kernel(xt, false, false), (unsigned)(mtiles * ntiles), kDqGemmThreads, st, xh, codes,
                  scales, M, N, K, lgB, y, mtiles, ntiles, 1);
  }
  // few rows: small tiles, and K split across workgroups (partial tiles added
  // into a zeroed y) when the tiles alone cannot fill the GPU
  const int64_t mtiles = (M + kDqGemmSmallTile - 1) / kDqGemmSmallTile;
  const int64_t ntiles = (N + kDqGemmSmallTile - 1) / kDqGemmSmallTile;
  const int64_t tiles = mtiles * ntiles, ksteps = K / kDqGemmK;
  int64_t splits = (kDqGemmSplitTarget + tiles - 1) / tiles;
  if (splits > ksteps) splits = ksteps;
  if (splits < 1) splits = 1;
  if (tiles * splits > kMaxGrid) return ZQ_E_SIZE;
  if (splits == 1)
    return launch(dqgemm_kernel(xt, true, false), (unsigned)tiles, kDqGemmSmallThreads, st, xh, codes, scales, M, N,
                  K, lgB, y, mtiles, ntiles, 1);
  const int64_t count = M * N, fill_grid = count / 256 + 1 < 4096 ? count / 256 + 1 : 4096;
  int rc = launch(fill_zero_kernel(), (unsigned)fill_grid, 256u, st, y, count);
  if (rc != ZQ_OK) return rc;
  return launch(dqgemm_kernel(xt, true, true), (unsigned)(tiles * splits), kDqGemmSmallThreads, st, xh, codes,
                scales, M, N, K, lgB, y, mtiles, ntiles, (int)splits);
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
