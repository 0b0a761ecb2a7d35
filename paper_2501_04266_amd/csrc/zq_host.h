// zq_host.h -- host-side helpers shared by the library's entry points:
// argument checks (block sizes, alignment, aliasing), grid sizing and kernel
// launches with the kernel's exact parameter types.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <initializer_list>
#include <tuple>
#include <utility>

#include "zq.h"

namespace zq {

constexpr int64_t kMaxGrid = 0x7fffffff;  // workgroups per launch

// Workgroups to cover `units` at `units_per_wg` each (0 if it exceeds the
// launch limit; callers turn that into ZQ_E_SIZE before anything is enqueued).
inline int64_t grid_for(int64_t units, int64_t units_per_wg) {
  int64_t g = (units + units_per_wg - 1) / units_per_wg;
  if (g < 1) g = 1;
  return g > kMaxGrid ? 0 : g;
}

// Launch with the kernel's exact parameter types; returns ZQ_E_HIP when the
// runtime rejects the launch.
template <typename... KArgs, typename... Args>
inline int launch(void (*kern)(KArgs...), unsigned grid, unsigned block, hipStream_t st, Args&&... args) {
  std::tuple<KArgs...> tup(std::forward<Args>(args)...);
  void* argv[sizeof...(KArgs)];
  std::apply([&](auto&... a) {
    int i = 0;
    ((argv[i++] = static_cast<void*>(&a)), ...);
  }, tup);
  hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(kern), dim3(grid), dim3(block), argv, 0, st);
  return e == hipSuccess ? ZQ_OK : ZQ_E_HIP;
}

inline int log2_block(int32_t block) {
  if (block < 32 || block > 1024 || (block & (block - 1)) != 0) return -1;
  int lg = 0;
  while ((1 << lg) < block) ++lg;
  return lg;
}

inline bool dtype_ok(int dt) { return dt == ZQ_F32 || dt == ZQ_F16 || dt == ZQ_BF16; }
inline int64_t elem_bytes(int dt) { return dt == ZQ_F32 ? 4 : 2; }
inline bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

struct Range {
  const void* p;
  int64_t bytes;
};
inline bool overlap(Range a, Range b) {
  uintptr_t a0 = reinterpret_cast<uintptr_t>(a.p), b0 = reinterpret_cast<uintptr_t>(b.p);
  return a0 < b0 + (uintptr_t)b.bytes && b0 < a0 + (uintptr_t)a.bytes;
}
inline bool any_overlap(std::initializer_list<Range> outs, std::initializer_list<Range> ins) {
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

inline int64_t num_scales(int64_t n, int32_t block) { return (n + block - 1) / block; }

}  // namespace zq
