// zq_probe.hip -- bandwidth ceilings for the benchmark (libzq_probe.so).
//
// Not part of the compression path: these kernels move bytes in the access
// patterns of the codec kernels with no arithmetic beyond an XOR, so their
// rates are the practical HBM ceilings the codec kernels are compared with.
// Same launch style as the codec kernels: 256 threads, whole-tensor grids (no
// grid-stride loop), 16 bytes per lane per access with consecutive lanes on
// consecutive 16-byte chunks, nontemporal loads and stores.  Chunks per
// thread are each pattern's fastest in a sweep of 1, 2, 4 and 8 (2 GiB,
// MI355X): copy and write one (6.5 and 6.7-6.9 TB/s, against 5.9 and 5.8
// with four), read four (7.0-7.2 TB/s for any count).
//
//   zqp_copy     dst[i] = src[i]                       (1 read stream, 1 write)
//   zqp_read     XOR of src, stored only if it equals a value the caller
//                passes (never, in practice), so the loads cannot be removed
//   zqp_write    dst[i] = pattern                      (1 write stream)
//   zqp_streams  dst[i] = XOR over p of src[p * slice + i]: the reduce level's
//                pattern (P read streams of slice_bytes, back to back, and one
//                write stream of slice_bytes)
//   zqp_expand   each thread loads 8 bytes and stores 16: the INT8 -> 16-bit
//                dequantiser's pattern (one read stream, a write stream twice
//                its size)
//
// Sizes are bytes and must be multiples of 16; pointers 16-byte aligned.
// Every call returns 0, or -1 on a bad argument (checked before any launch),
// or -7 when the launch fails.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
constexpr int kThreads = 256;
constexpr int kCopyChunks = 1, kReadChunks = 4, kWriteChunks = 1;  // 16-byte chunks per thread

__device__ __forceinline__ u32x4 ldnt(const u32x4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ u32x2 ldnt(const u32x2* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void stnt(u32x4* p, u32x4 v) { __builtin_nontemporal_store(v, p); }

// chunk u of thread t in workgroup g: index (g * C + u) * kThreads + t, C the
// pattern's chunks per thread
__global__ void __launch_bounds__(kThreads) k_copy(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                  int64_t n16) {
  constexpr int C = kCopyChunks;
  const int64_t base = (int64_t)blockIdx.x * C * kThreads + threadIdx.x;
  u32x4 v[C];
#pragma unroll
  for (int u = 0; u < C; ++u)
    if (base + u * kThreads < n16) v[u] = ldnt(src + base + u * kThreads);
#pragma unroll
  for (int u = 0; u < C; ++u)
    if (base + u * kThreads < n16) stnt(dst + base + u * kThreads, v[u]);
}

__global__ void __launch_bounds__(kThreads) k_read(const u32x4* __restrict__ src, int64_t n16, u32x4* sink,
                                                  uint32_t never) {
  constexpr int C = kReadChunks;
  const int64_t base = (int64_t)blockIdx.x * C * kThreads + threadIdx.x;
  u32x4 acc = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int u = 0; u < C; ++u)
    if (base + u * kThreads < n16) acc ^= ldnt(src + base + u * kThreads);
  if (acc.x == never && acc.y == never && acc.z == never && acc.w == never) *sink = acc;
}

__global__ void __launch_bounds__(kThreads) k_write(u32x4* __restrict__ dst, int64_t n16, uint32_t pattern) {
  constexpr int C = kWriteChunks;
  const int64_t base = (int64_t)blockIdx.x * C * kThreads + threadIdx.x;
  const u32x4 v = {pattern, pattern, pattern, pattern};
#pragma unroll
  for (int u = 0; u < C; ++u)
    if (base + u * kThreads < n16) stnt(dst + base + u * kThreads, v);
}

// one 16-byte chunk of every slice per thread, slices loaded 8 at a time
__global__ void __launch_bounds__(kThreads) k_streams(const u32x4* __restrict__ src, int P, int64_t slice16,
                                                     u32x4* __restrict__ dst) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= slice16) return;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (int p0 = 0; p0 < P; p0 += 8) {
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (p0 + u < P) v[u] = ldnt(src + (int64_t)(p0 + u) * slice16 + i);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (p0 + u < P) acc ^= v[u];
  }
  stnt(dst + i, acc);
}

// thread i: 8 bytes in at i, 16 bytes out at i (the dequantiser's one tile
// per wave, each store instruction covering 1 KiB)
__global__ void __launch_bounds__(kThreads) k_expand(const u32x2* __restrict__ src, int64_t n8,
                                                    u32x4* __restrict__ dst) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= n8) return;
  const u32x2 v = ldnt(src + i);
  stnt(dst + i, u32x4{v.x ^ 0x55555555u, v.x, v.y ^ 0x33333333u, v.y});
}

bool ok16(const void* p, int64_t bytes) {
  return p != nullptr && (reinterpret_cast<uintptr_t>(p) & 15) == 0 && bytes > 0 && bytes % 16 == 0;
}

int status() { return hipGetLastError() == hipSuccess ? 0 : -7; }

unsigned grid_of(int64_t n16, int64_t per_wg) { return (unsigned)((n16 + per_wg - 1) / per_wg); }

}  // namespace

extern "C" {

int zqp_copy(const void* src, void* dst, int64_t bytes, void* stream) {
  if (!ok16(src, bytes) || !ok16(dst, bytes) || bytes / 16 / (kCopyChunks * kThreads) >= 0x7fffffff) return -1;
  const int64_t n16 = bytes / 16;
  hipLaunchKernelGGL(k_copy, dim3(grid_of(n16, kCopyChunks * kThreads)), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), n16);
  return status();
}

int zqp_read(const void* src, int64_t bytes, void* sink, uint32_t never, void* stream) {
  if (!ok16(src, bytes) || !ok16(sink, 16) || bytes / 16 / (kReadChunks * kThreads) >= 0x7fffffff) return -1;
  const int64_t n16 = bytes / 16;
  hipLaunchKernelGGL(k_read, dim3(grid_of(n16, kReadChunks * kThreads)), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4*>(src), n16, static_cast<u32x4*>(sink),
                     never);
  return status();
}

int zqp_write(void* dst, int64_t bytes, uint32_t pattern, void* stream) {
  if (!ok16(dst, bytes) || bytes / 16 / (kWriteChunks * kThreads) >= 0x7fffffff) return -1;
  const int64_t n16 = bytes / 16;
  hipLaunchKernelGGL(k_write, dim3(grid_of(n16, kWriteChunks * kThreads)), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<u32x4*>(dst), n16, pattern);
  return status();
}

int zqp_streams(const void* src, int32_t P, int64_t slice_bytes, void* dst, void* stream) {
  if (P < 1 || P > 1024 || !ok16(src, slice_bytes) || !ok16(dst, slice_bytes) ||
      slice_bytes / 16 / kThreads >= 0x7fffffff)
    return -1;
  const int64_t slice16 = slice_bytes / 16;
  hipLaunchKernelGGL(k_streams, dim3(grid_of(slice16, kThreads)), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                     static_cast<const u32x4*>(src), (int)P, slice16, static_cast<u32x4*>(dst));
  return status();
}

int zqp_expand(const void* src, int64_t in_bytes, void* dst, void* stream) {
  if (!ok16(src, in_bytes) || !ok16(dst, 2 * in_bytes) || in_bytes / 8 / kThreads >= 0x7fffffff) return -1;
  const int64_t n8 = in_bytes / 8;
  hipLaunchKernelGGL(k_expand, dim3(grid_of(n8, kThreads)), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                     static_cast<const u32x2*>(src), n8, static_cast<u32x4*>(dst));
  return status();
}

}  // extern "C"
