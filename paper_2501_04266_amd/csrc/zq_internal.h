// zq_internal.h -- kernel handles shared between the kernel and API units.
#pragma once
#include <stdint.h>

namespace zq {

constexpr int kThreads = 256;  // threads per workgroup of the streaming kernels (4 waves)

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
