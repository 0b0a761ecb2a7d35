// zq_kernels.hip -- gfx950 kernels of the qwZ / qgZ compression path.
//
// Block-wise symmetric quantisation as ZeRO++ applies it to the weight
// Allgather (INT8) and the gradient all-to-all reduce-scatter (INT4), per the
// paper's Background (ZeRO++ subsection) and Design (Weight / Gradient
// Partitioning).  The exact definition every kernel reproduces bit for bit is
// written out in include/zq.h.
//
// All kernels are streaming, HBM-bound work (no contraction, so no MFMA):
//   * wave64 tiles with 16-byte loads/stores per lane, consecutive lanes on
//     consecutive addresses;
//   * per-block absmax reduced across the lanes of a block with DPP row
//     permutes (quad_perm, row_half_mirror, row_mirror) -- no LDS round trip;
//   * rounding to nearest-even by adding 1.5*2^23, which leaves the code as
//     two's complement in the low mantissa bits, then byte/nibble packing
//     with v_perm_b32;
//   * grid-stride loops over wave tiles; every wave of a launch runs the same
//     number of iterations, so cross-lane ops always see full waves.
//
// Floating point: built with -ffp-contract=off (and the pragma below) so a*b+c
// is never fused; fp32 division is the correctly rounded sequence; fp32 and
// fp16 denormals are preserved (default HIP mode).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "zq.h"
#include "zq_internal.h"

#pragma clang fp contract(off)

namespace zq {
namespace {

constexpr float kRoundMagic = 12582912.0f;  // 1.5 * 2^23
constexpr float kFlushBelow = 0x1p-119f;    // absmax below this: zero block

__device__ __forceinline__ uint32_t f2u(float f) { return __builtin_bit_cast(uint32_t, f); }
__device__ __forceinline__ float u2f(uint32_t u) { return __builtin_bit_cast(float, u); }

// fl(fl(v * r) + 1.5*2^23): for |fl(v*r)| < 2^22 the sum lies in [2^23, 2^24)
// where binary32 spacing is 1, so it is 1.5*2^23 + rint_even(fl(v*r)); the
// integer sits in the low mantissa bits as two's complement.
__device__ __forceinline__ uint32_t code_bits(float v, float r) {
  float t = v * r;
  return f2u(t + kRoundMagic);
}

// INT4 code (two's complement nibble k of w) as float.
__device__ __forceinline__ float nib_to_f32(uint32_t w, int k) {
  return (float)((int32_t)(w << (28 - 4 * k)) >> 28);
}

// Max over the L lanes of an aligned lane group (L a power of two <= 64).
// Non-negative binary32 values order like their bit patterns.
template <int L>
__device__ __forceinline__ uint32_t group_max(uint32_t v) {
  static_assert(L >= 1 && L <= 64 && (L & (L - 1)) == 0, "lane group");
  if constexpr (L >= 2) v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  if constexpr (L >= 4) v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  if constexpr (L >= 8) v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));  // row_half_mirror
  if constexpr (L >= 16) v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false)); // row_mirror
  if constexpr (L >= 32) v = max(v, (uint32_t)__shfl_xor((int)v, 16, 64));
  if constexpr (L >= 64) v = max(v, (uint32_t)__shfl_xor((int)v, 32, 64));
  return v;
}

__device__ __forceinline__ uint32_t wave_max(uint32_t v) { return group_max<64>(v); }

// byte 0 of m0..m3 -> bytes 0..3
__device__ __forceinline__ uint32_t pack_bytes4(uint32_t m0, uint32_t m1, uint32_t m2, uint32_t m3) {
  uint32_t lo = __builtin_amdgcn_perm(m1, m0, 0x0c0c0400u);
  uint32_t hi = __builtin_amdgcn_perm(m3, m2, 0x0c0c0400u);
  return __builtin_amdgcn_perm(hi, lo, 0x05040100u);
}

// low nibble of m[0..7] -> nibbles 0..7 (element 2j low, 2j+1 high of byte j)
__device__ __forceinline__ uint32_t pack_nibbles8(const uint32_t* m) {
  uint32_t ev = pack_bytes4(m[0], m[2], m[4], m[6]);
  uint32_t od = pack_bytes4(m[1], m[3], m[5], m[7]);
  return (ev & 0x0f0f0f0fu) | ((od << 4) & 0xf0f0f0f0u);
}

// ------------------------------------------------------------------ element I/O

template <int DT>
struct Elem;

template <>
struct Elem<ZQ_F32> {
  __device__ static void load16(const void* p, int64_t i, float (&v)[16]) {
    const float4* q = reinterpret_cast<const float4*>(static_cast<const float*>(p) + i);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float4 f = q[k];
      v[4 * k] = f.x; v[4 * k + 1] = f.y; v[4 * k + 2] = f.z; v[4 * k + 3] = f.w;
    }
  }
  __device__ static float load1(const void* p, int64_t i) { return static_cast<const float*>(p)[i]; }
  __device__ static void store16(void* p, int64_t i, const float (&v)[16]) {
    float4* q = reinterpret_cast<float4*>(static_cast<float*>(p) + i);
#pragma unroll
    for (int k = 0; k < 4; ++k) q[k] = make_float4(v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3]);
  }
  __device__ static void store1(void* p, int64_t i, float v) { static_cast<float*>(p)[i] = v; }
};

// bf16 <-> f32: widening is a 16-bit shift; narrowing is v_cvt_pk_bf16_f32
// (round to nearest even).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t bf16x2_bits(float a, float b) {
  f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

template <>
struct Elem<ZQ_BF16> {
  __device__ static void load16(const void* p, int64_t i, float (&v)[16]) {
    const uint4* q = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p) + i);
    uint4 a = q[0], b = q[1];
    uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      v[2 * k] = u2f(w[k] << 16);
      v[2 * k + 1] = u2f(w[k] & 0xffff0000u);
    }
  }
  __device__ static float load1(const void* p, int64_t i) {
    return u2f((uint32_t)static_cast<const uint16_t*>(p)[i] << 16);
  }
  __device__ static void store16(void* p, int64_t i, const float (&v)[16]) {
    uint4* q = reinterpret_cast<uint4*>(static_cast<uint16_t*>(p) + i);
    q[0] = make_uint4(bf16x2_bits(v[0], v[1]), bf16x2_bits(v[2], v[3]), bf16x2_bits(v[4], v[5]), bf16x2_bits(v[6], v[7]));
    q[1] = make_uint4(bf16x2_bits(v[8], v[9]), bf16x2_bits(v[10], v[11]), bf16x2_bits(v[12], v[13]), bf16x2_bits(v[14], v[15]));
  }
  __device__ static void store1(void* p, int64_t i, float v) {
    static_cast<uint16_t*>(p)[i] = (uint16_t)(bf16x2_bits(v, 0.0f) & 0xffffu);
  }
};

__device__ __forceinline__ float h2f(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}
// binary32 -> binary16, nearest even (v_cvt_f16_f32).  The empty asm pins v
// as a materialised binary32 value: without it the compiler folds a preceding
// fp32 multiply and this narrowing into one v_fma_mixlo_f16, which rounds the
// exact product once instead of rounding it to binary32 first.
__device__ __forceinline__ uint32_t f2h(float v) {
  asm("" : "+v"(v));
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v);
}

template <>
struct Elem<ZQ_F16> {
  __device__ static void load16(const void* p, int64_t i, float (&v)[16]) {
    const uint4* q = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p) + i);
    uint4 a = q[0], b = q[1];
    uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      v[2 * k] = h2f(w[k] & 0xffffu);
      v[2 * k + 1] = h2f(w[k] >> 16);
    }
  }
  __device__ static float load1(const void* p, int64_t i) { return h2f(static_cast<const uint16_t*>(p)[i]); }
  __device__ static void store16(void* p, int64_t i, const float (&v)[16]) {
    uint4* q = reinterpret_cast<uint4*>(static_cast<uint16_t*>(p) + i);
    uint32_t w[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) w[k] = f2h(v[2 * k]) | (f2h(v[2 * k + 1]) << 16);
    q[0] = make_uint4(w[0], w[1], w[2], w[3]);
    q[1] = make_uint4(w[4], w[5], w[6], w[7]);
  }
  __device__ static void store1(void* p, int64_t i, float v) { static_cast<uint16_t*>(p)[i] = (uint16_t)f2h(v); }
};

__device__ __forceinline__ int64_t wave_id() {
  return (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
}
__device__ __forceinline__ int64_t wave_count() { return (int64_t)gridDim.x * (blockDim.x >> 6); }

}  // namespace

// ------------------------------------------------------------------ quantise
// Full blocks only.  A lane owns 16 consecutive elements; L = B/16 lanes hold
// one block; a wave tile is 64/L blocks.

template <int DT, int QBITS, int B>
__global__ void __launch_bounds__(kThreads) k_quantize(const void* __restrict__ x, int64_t nfull,
                                                       uint8_t* __restrict__ out, float* __restrict__ scales) {
  constexpr int E = 16, L = B / E, BPW = 64 / L;
  constexpr float QMAX = QBITS == 8 ? 127.0f : 7.0f;
  const int lane = threadIdx.x & 63;
  const int64_t ntiles = (nfull + BPW - 1) / BPW;
  for (int64_t t = wave_id(); t < ntiles; t += wave_count()) {
    const int64_t blk = t * BPW + lane / L;
    const bool valid = blk < nfull;
    const int64_t e0 = blk * B + (int64_t)(lane % L) * E;
    float v[E];
    if (valid) {
      Elem<DT>::load16(x, e0, v);
    } else {
#pragma unroll
      for (int k = 0; k < E; ++k) v[k] = 0.0f;
    }
    float a = fabsf(v[0]);
#pragma unroll
    for (int k = 1; k < E; ++k) a = fmaxf(a, fabsf(v[k]));
    const float amax = u2f(group_max<L>(f2u(a)));
    float s = 0.0f, r = 0.0f;
    if (amax >= kFlushBelow) {
      s = amax / QMAX;
      r = QMAX / amax;
    }
    uint32_t m[E];
#pragma unroll
    for (int k = 0; k < E; ++k) m[k] = code_bits(v[k], r);
    if (valid) {
      if constexpr (QBITS == 8) {
        uint4 o = make_uint4(pack_bytes4(m[0], m[1], m[2], m[3]), pack_bytes4(m[4], m[5], m[6], m[7]),
                             pack_bytes4(m[8], m[9], m[10], m[11]), pack_bytes4(m[12], m[13], m[14], m[15]));
        *reinterpret_cast<uint4*>(out + e0) = o;
      } else {
        uint2 o = make_uint2(pack_nibbles8(m), pack_nibbles8(m + 8));
        *reinterpret_cast<uint2*>(out + (e0 >> 1)) = o;
      }
      if (lane % L == 0) scales[blk] = s;
    }
  }
}

// The one short block [start, start + len), len < B <= 1024; one wave.
template <int DT, int QBITS>
__global__ void __launch_bounds__(64) k_quantize_tail(const void* __restrict__ x, int64_t start, int len,
                                                      uint8_t* __restrict__ out, float* __restrict__ scale) {
  constexpr float QMAX = QBITS == 8 ? 127.0f : 7.0f;
  const int lane = threadIdx.x;
  float a = 0.0f;
  for (int j = lane; j < len; j += 64) a = fmaxf(a, fabsf(Elem<DT>::load1(x, start + j)));
  const float amax = u2f(wave_max(f2u(a)));
  float s = 0.0f, r = 0.0f;
  if (amax >= kFlushBelow) {
    s = amax / QMAX;
    r = QMAX / amax;
  }
  if constexpr (QBITS == 8) {
    for (int j = lane; j < len; j += 64) out[start + j] = (uint8_t)code_bits(Elem<DT>::load1(x, start + j), r);
  } else {
    for (int k = lane; 2 * k < len; k += 64) {
      uint32_t lo = code_bits(Elem<DT>::load1(x, start + 2 * k), r);
      uint32_t hi = (2 * k + 1 < len) ? code_bits(Elem<DT>::load1(x, start + 2 * k + 1), r) : 0u;
      out[(start >> 1) + k] = (uint8_t)((lo & 0xfu) | ((hi & 0xfu) << 4));
    }
  }
  if (lane == 0) *scale = s;
}

// ------------------------------------------------------------------ INT8 dequantise
// A thread owns 16 consecutive codes (one 16-byte load), all in one block.

template <int DT>
__global__ void __launch_bounds__(kThreads) k_qwz_dequant(const int8_t* __restrict__ codes,
                                                          const float* __restrict__ scales, int64_t n, int lgB,
                                                          void* __restrict__ y) {
  const int64_t ngroups = n >> 4;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t nthreads = (int64_t)gridDim.x * blockDim.x;
  for (int64_t g = tid; g < ngroups; g += nthreads) {
    const int64_t e0 = g << 4;
    const uint4 w4 = *reinterpret_cast<const uint4*>(codes + e0);
    const float s = scales[e0 >> lgB];
    const uint32_t w[4] = {w4.x, w4.y, w4.z, w4.w};
    float v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) v[k] = (float)(int32_t)(int8_t)(w[k >> 2] >> (8 * (k & 3))) * s;
    Elem<DT>::store16(y, e0, v);
  }
  const int64_t rest = n - (ngroups << 4);
  if (tid < rest) {
    const int64_t i = (ngroups << 4) + tid;
    Elem<DT>::store1(y, i, (float)(int32_t)codes[i] * scales[i >> lgB]);
  }
}

// ------------------------------------------------------------------ INT4 dequantise
// A thread owns 16 consecutive nibbles (one 8-byte load).

template <int DT>
__global__ void __launch_bounds__(kThreads) k_qgz_dequant(const uint8_t* __restrict__ packed,
                                                          const float* __restrict__ scales, int64_t n, int lgB,
                                                          void* __restrict__ y) {
  const int64_t ngroups = n >> 4;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t nthreads = (int64_t)gridDim.x * blockDim.x;
  for (int64_t g = tid; g < ngroups; g += nthreads) {
    const int64_t e0 = g << 4;
    const uint2 w2 = *reinterpret_cast<const uint2*>(packed + (e0 >> 1));
    const float s = scales[e0 >> lgB];
    float v[16];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = nib_to_f32(w2.x, k) * s;
#pragma unroll
    for (int k = 0; k < 8; ++k) v[8 + k] = nib_to_f32(w2.y, k) * s;
    Elem<DT>::store16(y, e0, v);
  }
  const int64_t rest = n - (ngroups << 4);
  if (tid < rest) {
    const int64_t i = (ngroups << 4) + tid;
    const uint32_t byte = packed[i >> 1];
    Elem<DT>::store1(y, i, nib_to_f32(byte, (int)(i & 1)) * scales[i >> lgB]);
  }
}

// ------------------------------------------------------------------ reduce level
// Fast path: slices 16-byte aligned (m % 32 == 0), full blocks only.  A lane
// owns 32 consecutive elements (16 bytes of every slice); L = B/32 lanes hold
// one block.  Slices are summed in ascending order, exactly as defined.

template <int B>
__global__ void __launch_bounds__(kThreads) k_reduce(const uint8_t* __restrict__ in, const float* __restrict__ sin,
                                                     int P, int64_t slice_bytes, int64_t slice_scales,
                                                     int64_t nfull, uint8_t* __restrict__ out,
                                                     float* __restrict__ sout) {
  constexpr int E = 32, L = B / E, BPW = 64 / L, U = 4;
  const int lane = threadIdx.x & 63;
  const int64_t ntiles = (nfull + BPW - 1) / BPW;
  for (int64_t t = wave_id(); t < ntiles; t += wave_count()) {
    const int64_t blk = t * BPW + lane / L;
    const bool valid = blk < nfull;
    const int64_t byte0 = (blk * B + (int64_t)(lane % L) * E) >> 1;
    float acc[E];
#pragma unroll
    for (int k = 0; k < E; ++k) acc[k] = 0.0f;
    for (int p0 = 0; p0 < P; p0 += U) {
      uint4 w[U];
      float s[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int p = p0 + u;
        if (valid && p < P) {
          w[u] = *reinterpret_cast<const uint4*>(in + (int64_t)p * slice_bytes + byte0);
          s[u] = sin[(int64_t)p * slice_scales + blk];
        } else {
          w[u] = make_uint4(0u, 0u, 0u, 0u);
          s[u] = 0.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (p0 + u < P) {
          const uint32_t ww[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
#pragma unroll
          for (int k = 0; k < E; ++k) {
            const float prod = nib_to_f32(ww[k >> 3], k & 7) * s[u];
            acc[k] = acc[k] + prod;
          }
        }
      }
    }
    float a = fabsf(acc[0]);
#pragma unroll
    for (int k = 1; k < E; ++k) a = fmaxf(a, fabsf(acc[k]));
    const float amax = u2f(group_max<L>(f2u(a)));
    float so = 0.0f, r = 0.0f;
    if (amax >= kFlushBelow) {
      so = amax / 7.0f;
      r = 7.0f / amax;
    }
    uint32_t m[E];
#pragma unroll
    for (int k = 0; k < E; ++k) m[k] = code_bits(acc[k], r);
    if (valid) {
      *reinterpret_cast<uint4*>(out + byte0) =
          make_uint4(pack_nibbles8(m), pack_nibbles8(m + 8), pack_nibbles8(m + 16), pack_nibbles8(m + 24));
      if (lane % L == 0) sout[blk] = so;
    }
  }
}

// Generic path: any m, any slice alignment; one wave per block, blocks
// [blk_begin, blk_begin + gridDim.x).  A lane owns byte j = lane + 64 i of the
// block (elements 2j, 2j+1), i < B/128 rounded up.
__global__ void __launch_bounds__(64) k_reduce_generic(const uint8_t* __restrict__ in, const float* __restrict__ sin,
                                                       int P, int64_t slice_bytes, int64_t slice_scales, int64_t m,
                                                       int B, int64_t blk_begin, uint8_t* __restrict__ out,
                                                       float* __restrict__ sout) {
  constexpr int MAXI = 1024 / 128;
  const int lane = threadIdx.x;
  const int64_t blk = blk_begin + blockIdx.x;
  const int64_t base = blk * B;
  const int len = (int)((m - base) < B ? (m - base) : B);
  const int nbytes = (len + 1) >> 1;
  float acc[2 * MAXI];
#pragma unroll
  for (int k = 0; k < 2 * MAXI; ++k) acc[k] = 0.0f;
  for (int p = 0; p < P; ++p) {
    const float s = sin[(int64_t)p * slice_scales + blk];
    const uint8_t* src = in + (int64_t)p * slice_bytes + (base >> 1);
#pragma unroll
    for (int i = 0; i < MAXI; ++i) {
      const int j = lane + 64 * i;
      if (j < nbytes) {
        const uint32_t byte = src[j];
        acc[2 * i] = acc[2 * i] + nib_to_f32(byte, 0) * s;
        acc[2 * i + 1] = acc[2 * i + 1] + nib_to_f32(byte, 1) * s;
      }
    }
  }
  float a = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXI; ++i) {
    const int j = lane + 64 * i;
    if (j < nbytes) {
      a = fmaxf(a, fabsf(acc[2 * i]));
      if (2 * j + 1 < len) a = fmaxf(a, fabsf(acc[2 * i + 1]));
    }
  }
  const float amax = u2f(wave_max(f2u(a)));
  float so = 0.0f, r = 0.0f;
  if (amax >= kFlushBelow) {
    so = amax / 7.0f;
    r = 7.0f / amax;
  }
#pragma unroll
  for (int i = 0; i < MAXI; ++i) {
    const int j = lane + 64 * i;
    if (j < nbytes) {
      const uint32_t lo = code_bits(acc[2 * i], r);
      const uint32_t hi = (2 * j + 1 < len) ? code_bits(acc[2 * i + 1], r) : 0u;
      out[(base >> 1) + j] = (uint8_t)((lo & 0xfu) | ((hi & 0xfu) << 4));
    }
  }
  if (lane == 0) sout[blk] = so;
}

// ------------------------------------------------------------------ instantiation tables

template <int DT, int QB>
static QuantKernel quant_kernel_for(int lgB) {
  switch (lgB) {
    case 5: return &k_quantize<DT, QB, 32>;
    case 6: return &k_quantize<DT, QB, 64>;
    case 7: return &k_quantize<DT, QB, 128>;
    case 8: return &k_quantize<DT, QB, 256>;
    case 9: return &k_quantize<DT, QB, 512>;
    default: return &k_quantize<DT, QB, 1024>;
  }
}

QuantKernel quant_kernel(int dt, int qbits, int lgB) {
  if (qbits == 8) {
    if (dt == ZQ_F32) return quant_kernel_for<ZQ_F32, 8>(lgB);
    if (dt == ZQ_F16) return quant_kernel_for<ZQ_F16, 8>(lgB);
    return quant_kernel_for<ZQ_BF16, 8>(lgB);
  }
  if (dt == ZQ_F32) return quant_kernel_for<ZQ_F32, 4>(lgB);
  if (dt == ZQ_F16) return quant_kernel_for<ZQ_F16, 4>(lgB);
  return quant_kernel_for<ZQ_BF16, 4>(lgB);
}

QuantTailKernel quant_tail_kernel(int dt, int qbits) {
  if (qbits == 8) {
    if (dt == ZQ_F32) return &k_quantize_tail<ZQ_F32, 8>;
    if (dt == ZQ_F16) return &k_quantize_tail<ZQ_F16, 8>;
    return &k_quantize_tail<ZQ_BF16, 8>;
  }
  if (dt == ZQ_F32) return &k_quantize_tail<ZQ_F32, 4>;
  if (dt == ZQ_F16) return &k_quantize_tail<ZQ_F16, 4>;
  return &k_quantize_tail<ZQ_BF16, 4>;
}

Dequant8Kernel dequant8_kernel(int dt) {
  if (dt == ZQ_F32) return &k_qwz_dequant<ZQ_F32>;
  if (dt == ZQ_F16) return &k_qwz_dequant<ZQ_F16>;
  return &k_qwz_dequant<ZQ_BF16>;
}

Dequant4Kernel dequant4_kernel(int dt) {
  if (dt == ZQ_F32) return &k_qgz_dequant<ZQ_F32>;
  if (dt == ZQ_F16) return &k_qgz_dequant<ZQ_F16>;
  return &k_qgz_dequant<ZQ_BF16>;
}

ReduceKernel reduce_kernel(int lgB) {
  switch (lgB) {
    case 5: return &k_reduce<32>;
    case 6: return &k_reduce<64>;
    case 7: return &k_reduce<128>;
    case 8: return &k_reduce<256>;
    case 9: return &k_reduce<512>;
    default: return &k_reduce<1024>;
  }
}

ReduceGenericKernel reduce_generic_kernel() { return &k_reduce_generic; }

}  // namespace zq
