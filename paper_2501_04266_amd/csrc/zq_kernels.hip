// zq_kernels.hip -- gfx950 kernels of the qwZ / qgZ compression path.
//
// Block-wise symmetric quantisation as ZeRO++ applies it to the weight
// Allgather (INT8) and the gradient all-to-all reduce-scatter (INT4), per the
// paper's Background (ZeRO++ subsection) and Design (Weight / Gradient
// Partitioning).  The exact definition every kernel reproduces bit for bit is
// written out in include/zq.h.
//
// All kernels are streaming, HBM-bound work (no contraction, so no MFMA):
//   * one tile of 64 lanes x E elements per wave, launches covering the whole
//     tensor, nontemporal loads and stores (data is touched once);
//   * per-block absmax reduced across the lanes of a block with DPP row
//     permutes (quad_perm, row_half_mirror, row_mirror) -- no LDS round trip;
//   * rounding to nearest-even by adding 1.5*2^23, which leaves the code as
//     two's complement in the low mantissa bits, then byte/nibble packing
//     with v_perm_b32;
//   * the reduce level, the one kernel with real arithmetic per byte (P
//     multiplies and adds per output element), converts a nibble with one
//     v_cvt_off_f32_i4 (q/16 exactly) and multiplies by 16*s, which is exact,
//     so every product is still fl(q*s).
//
// Floating point: built with -ffp-contract=off (and the pragma below) so a*b+c
// is never fused; fp32 division is the correctly rounded sequence; fp32 and
// fp16 denormals are preserved (default HIP mode).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "zq.h"
#include "zq_device.h"
#include "zq_internal.h"

#pragma clang fp contract(off)

// Nontemporal hints per kernel family: bit 0 = loads, bit 1 = stores.  Data
// streamed once gains from them; a kernel whose input was just written by the
// previous call (the dequantiser after a reduce level) loses its cache hits.
// The quantisers: INT8 output measured faster with plain stores (the
// degree-2 half shard 100.3 against 104.9 us), INT4 output with nontemporal
// ones (the fp32 gradient 310.0 against 312.0 us).
// Wave priority while a wave issues its loads (s_setprio, within the
// kernel): raised so that the loads of a newly started wave go out ahead of
// other waves' arithmetic, then back to normal for the wave's own arithmetic.
#ifndef ZQ_PRIO_QUANT
#define ZQ_PRIO_QUANT 1
#endif
#ifndef ZQ_PRIO_REDUCE
#define ZQ_PRIO_REDUCE 0
#endif
#ifndef ZQ_PRIO_DEQ
#define ZQ_PRIO_DEQ 0
#endif
template <int ON>
__device__ __forceinline__ void prio_issue() {
  if constexpr (ON) __builtin_amdgcn_s_setprio(3);
}
template <int ON>
__device__ __forceinline__ void prio_compute() {
  if constexpr (ON) __builtin_amdgcn_s_setprio(0);
}
#ifndef ZQ_NT_QUANT8
#define ZQ_NT_QUANT8 1
#endif
#ifndef ZQ_NT_QUANT4
#define ZQ_NT_QUANT4 3
#endif
#ifndef ZQ_NT_DEQ8
#define ZQ_NT_DEQ8 3
#endif
#ifndef ZQ_NT_DEQ4
#define ZQ_NT_DEQ4 0
#endif
#ifndef ZQ_NT_REDUCE
#define ZQ_NT_REDUCE 3
#endif
// Dequantisers with more than 16 output bytes per thread stage them in LDS.
#ifndef ZQ_DEQ_STAGE
#define ZQ_DEQ_STAGE 1
#endif
// Scale arrays are written 4 bytes per block, i.e. in partial cache lines:
// plain stores let L2 merge them into full lines before write-back.
#ifndef ZQ_NT_SCALES
#define ZQ_NT_SCALES 0
#endif
// slices loaded ahead per batch in the reduce level (large / small levels)
#ifndef ZQ_REDUCE_U
#define ZQ_REDUCE_U 4
#endif
#ifndef ZQ_REDUCE_U_SMALL
#define ZQ_REDUCE_U_SMALL 16
#endif
// batch pipelining (see the reduce kernel) per launch shape: large / P <= 2 / small
#ifndef ZQ_REDUCE_PIPE
#define ZQ_REDUCE_PIPE 1
#endif
#ifndef ZQ_REDUCE_PIPE2
#define ZQ_REDUCE_PIPE2 1
#endif
#ifndef ZQ_REDUCE_PIPE_SMALL
#define ZQ_REDUCE_PIPE_SMALL 0
#endif

namespace zq {
namespace {


constexpr float kRoundMagic = 12582912.0f;  // 1.5 * 2^23
constexpr float kFlushBelow = 0x1p-119f;    // absmax below this: zero block
constexpr float kMaxFloat = 3.40282346638528859812e+38f;

template <int NT, typename T>
__device__ __forceinline__ T ld(const T* p) {
  if constexpr (NT & 1) return __builtin_nontemporal_load(p);
  else return *p;
}
template <int NT, typename T>
__device__ __forceinline__ void st(T* p, T v) {
  if constexpr (NT & 2) __builtin_nontemporal_store(v, p);
  else *p = v;
}


// fl(fl(v * r) + 1.5*2^23): for |fl(v*r)| < 2^22 the sum lies in [2^23, 2^24)
// where binary32 spacing is 1, so it is 1.5*2^23 + rint_even(fl(v*r)); the
// integer sits in the low mantissa bits as two's complement.
__device__ __forceinline__ uint32_t code_bits(float v, float r) {
  float t = v * r;
  return f2u(t + kRoundMagic);
}

// Block scale fl(a / qmax) for a normal a >= 2^-119, via one binary64
// multiply: a/qmax is either a binary32 value or lies at least
// ulp(a/qmax) / (2 qmax) >= (a/qmax) * 2^-32 away from every binary32 rounding
// boundary (qmax is odd, so a/qmax is not dyadic unless qmax divides a's
// significand), while a * fl64(1/qmax) is within 2^-52 relative of a/qmax.
// Rounding that to binary32 (nearest even) therefore gives fl(a / qmax),
// the correctly rounded quotient, in 3 instructions instead of a division.
template <int QMAX>
__device__ __forceinline__ float scale_of(float amax) {
  return (float)((double)amax * (1.0 / (double)QMAX));
}

// INT4 code (two's complement nibble k of w) as float.
__device__ __forceinline__ float nib_to_f32(uint32_t w, int k) {
  return (float)((int32_t)(w << (28 - 4 * k)) >> 28);
}

// q/16 for the two's-complement low nibble of byte BYTE of w, in one
// instruction (v_cvt_off_f32_i4 with an SDWA byte select).
template <int BYTE>
__device__ __forceinline__ float nib_over_16(uint32_t w) {
  float f;
  if constexpr (BYTE == 0)
    asm("v_cvt_off_f32_i4_sdwa %0, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0" : "=v"(f) : "v"(w));
  else if constexpr (BYTE == 1)
    asm("v_cvt_off_f32_i4_sdwa %0, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1" : "=v"(f) : "v"(w));
  else if constexpr (BYTE == 2)
    asm("v_cvt_off_f32_i4_sdwa %0, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2" : "=v"(f) : "v"(w));
  else
    asm("v_cvt_off_f32_i4_sdwa %0, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3" : "=v"(f) : "v"(w));
  return f;
}

// The 8 nibbles of w, each as q/16 (element order: low nibble of byte 0 first).
__device__ __forceinline__ void nibbles_over_16(uint32_t w, float* o) {
  const uint32_t h = w >> 4;
  o[0] = nib_over_16<0>(w); o[1] = nib_over_16<0>(h);
  o[2] = nib_over_16<1>(w); o[3] = nib_over_16<1>(h);
  o[4] = nib_over_16<2>(w); o[5] = nib_over_16<2>(h);
  o[6] = nib_over_16<3>(w); o[7] = nib_over_16<3>(h);
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

// ------------------------------------------------------------------ raw I/O

template <int NT, int NW>
__device__ __forceinline__ void load_words(const void* p, uint32_t (&w)[NW]) {
  if constexpr (NW % 4 == 0) {
#pragma unroll
    for (int k = 0; k < NW / 4; ++k) {
      const u32x4 t = ld<NT>(static_cast<const u32x4*>(p) + k);
      w[4 * k] = t.x; w[4 * k + 1] = t.y; w[4 * k + 2] = t.z; w[4 * k + 3] = t.w;
    }
  } else if constexpr (NW == 2) {
    const u32x2 t = ld<NT>(static_cast<const u32x2*>(p));
    w[0] = t.x; w[1] = t.y;
  } else {
    static_assert(NW == 1, "words");
    w[0] = ld<NT>(static_cast<const uint32_t*>(p));
  }
}

template <int NT, int NW>
__device__ __forceinline__ void store_words(void* p, const uint32_t (&w)[NW]) {
  if constexpr (NW % 4 == 0) {
#pragma unroll
    for (int k = 0; k < NW / 4; ++k)
      st<NT>(static_cast<u32x4*>(p) + k, u32x4{w[4 * k], w[4 * k + 1], w[4 * k + 2], w[4 * k + 3]});
  } else if constexpr (NW == 2) {
    st<NT>(static_cast<u32x2*>(p), u32x2{w[0], w[1]});
  } else {
    static_assert(NW == 1, "words");
    st<NT>(static_cast<uint32_t*>(p), w[0]);
  }
}

// ------------------------------------------------------------------ element formats

template <int DT>
constexpr int elem_size() { return DT == ZQ_F32 ? 4 : 2; }

// E consecutive elements from element index i, widened to binary32 (exact).
template <int NT, int DT, int E>
__device__ __forceinline__ void load_elems(const void* p, int64_t i, float (&v)[E]) {
  constexpr int NW = E * elem_size<DT>() / 4;
  uint32_t w[NW];
  load_words<NT, NW>(static_cast<const char*>(p) + i * elem_size<DT>(), w);
#pragma unroll
  for (int k = 0; k < NW; ++k) {
    if constexpr (DT == ZQ_F32) {
      v[k] = u2f(w[k]);
    } else if constexpr (DT == ZQ_BF16) {
      v[2 * k] = u2f(w[k] << 16);
      v[2 * k + 1] = u2f(w[k] & 0xffff0000u);
    } else {
      v[2 * k] = h2f(w[k] & 0xffffu);
      v[2 * k + 1] = h2f(w[k] >> 16);
    }
  }
}

// E binary32 values narrowed (nearest even) and stored from element index i.
template <int NT, int DT, int E>
__device__ __forceinline__ void store_elems(void* p, int64_t i, const float (&v)[E]) {
  constexpr int NW = E * elem_size<DT>() / 4;
  uint32_t w[NW];
#pragma unroll
  for (int k = 0; k < NW; ++k) {
    if constexpr (DT == ZQ_F32) w[k] = f2u(v[k]);
    else if constexpr (DT == ZQ_BF16) w[k] = bf16x2_bits(v[2 * k], v[2 * k + 1]);
    else w[k] = f2h(v[2 * k]) | (f2h(v[2 * k + 1]) << 16);
  }
  store_words<NT, NW>(static_cast<char*>(p) + i * elem_size<DT>(), w);
}

template <int DT>
__device__ __forceinline__ float load1(const void* p, int64_t i) {
  if constexpr (DT == ZQ_F32) return static_cast<const float*>(p)[i];
  else if constexpr (DT == ZQ_BF16) return u2f((uint32_t)static_cast<const uint16_t*>(p)[i] << 16);
  else return h2f(static_cast<const uint16_t*>(p)[i]);
}

template <int DT>
__device__ __forceinline__ void store1(void* p, int64_t i, float v) {
  if constexpr (DT == ZQ_F32) static_cast<float*>(p)[i] = v;
  else if constexpr (DT == ZQ_BF16) static_cast<uint16_t*>(p)[i] = (uint16_t)(bf16x2_bits(v, 0.0f) & 0xffffu);
  else static_cast<uint16_t*>(p)[i] = (uint16_t)f2h(v);
}


}  // namespace

// ------------------------------------------------------------------ quantise
// Full blocks only.  A lane owns E elements of one block, as C = E*size/16
// chunks of 16 bytes: L = B/E lanes hold the block, and chunk j of the
// block's lane i is the block's chunk j*L + i, so each load instruction of a
// wave reads whole runs of L*16 bytes while the block's absmax, scale and
// reciprocal are computed once per lane for all E elements.  One wave tile
// is 64/L blocks; a workgroup's tiles are adjacent.  The codes and scales of
// a workgroup are staged in LDS and written back as one contiguous run of
// 16-byte stores: at this kernel's ~8:1 read:write mix
// that keeps the write stream from slowing the reads (per-lane 2-byte stores
// measured ~10% slower).  A workgroup holding the last, partial tile stores
// straight from its lanes instead.  When n is not a multiple of B, one more
// workgroup quantises the short last block, in the same launch.

// The one short block [start, start + len), len < B <= 1024, quantised by
// one wave; the scale goes to *scale.
template <int DT, int QBITS>
__device__ __forceinline__ void quantize_tail(const void* __restrict__ x, int64_t start, int len,
                                              uint8_t* __restrict__ out, float* __restrict__ scale) {
  constexpr float QMAX = QBITS == 8 ? 127.0f : 7.0f;
  const int lane = threadIdx.x & 63;
  float a = 0.0f;
  for (int j = lane; j < len; j += 64) a = fmaxf(a, fabsf(load1<DT>(x, start + j)));
  const float amax = u2f(wave_max(f2u(a)));
  float s = 0.0f, r = 0.0f;
  if (amax >= kFlushBelow) {
    s = scale_of<(int)QMAX>(amax);
    r = QMAX / amax;
  }
  if constexpr (QBITS == 8) {
    for (int j = lane; j < len; j += 64) out[start + j] = (uint8_t)code_bits(load1<DT>(x, start + j), r);
  } else {
    for (int k = lane; 2 * k < len; k += 64) {
      uint32_t lo = code_bits(load1<DT>(x, start + 2 * k), r);
      uint32_t hi = (2 * k + 1 < len) ? code_bits(load1<DT>(x, start + 2 * k + 1), r) : 0u;
      out[(start >> 1) + k] = (uint8_t)((lo & 0xfu) | ((hi & 0xfu) << 4));
    }
  }
  if (lane == 0) *scale = s;
}

template <int DT, int QBITS, int B>
__global__ void __launch_bounds__(kQuantThreads) k_quantize(const void* __restrict__ x, int64_t nfull,
                                                            uint8_t* __restrict__ out, float* __restrict__ scales,
                                                            int tail) {
  constexpr int E = quant_elems(elem_size<DT>(), B), L = B / E, BPW = 64 / L;
  constexpr int CE = 16 / elem_size<DT>(), C = E / CE;          // elements per chunk, chunks per lane
  constexpr int T = quant_tiles(elem_size<DT>()), WAVES = kQuantThreads / 64;
  constexpr float QMAX = QBITS == 8 ? 127.0f : 7.0f;
  constexpr int NT = QBITS == 8 ? ZQ_NT_QUANT8 : ZQ_NT_QUANT4;
  constexpr int OB = QBITS == 8 ? E : E / 2;                    // code bytes per lane and tile
  constexpr int OBC = OB / C;                                   // code bytes per chunk
  constexpr int BB = B * OB / E;                                // code bytes per block
  constexpr int WG_BLOCKS = WAVES * T * BPW;                    // blocks per workgroup
  constexpr int WG_BYTES = WAVES * T * 64 * OB;                 // code bytes per workgroup
  constexpr int NWO = OB >= 4 ? OB / 4 : 1;
  static_assert(E % CE == 0 && L >= 1 && L <= 64 && WG_BYTES % 16 == 0, "lane layout");
  static_assert(OBC == 2 || OBC % 4 == 0, "chunk codes");
  __shared__ u32x4 obuf[WG_BYTES / 16];
  __shared__ float sbuf[WG_BLOCKS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // with a short last block (tail > 0 elements) the launch has one workgroup
  // more than the full blocks need: the last one quantises that block with
  // its first wave (scalar test: 32-bit workgroup indices)
  if (tail > 0 && blockIdx.x == gridDim.x - 1) {
    if (wave == 0) quantize_tail<DT, QBITS>(x, nfull * B, tail, out, scales + nfull);
    return;
  }
  // workgroup g owns tiles [g*WAVES*T, (g+1)*WAVES*T); its t-th round of loads
  // covers WAVES adjacent tiles, one per wave
  const int64_t wg_blk0 = (int64_t)blockIdx.x * WG_BLOCKS;
  const int li = lane % L;  // the lane's index within its block
  prio_issue<ZQ_PRIO_QUANT>();
  float v[T][E];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int64_t blk = wg_blk0 + (t * WAVES + wave) * BPW + lane / L;
#pragma unroll
    for (int j = 0; j < C; ++j) {
      float c[CE];
      if (blk < nfull) {
        load_elems<NT, DT, CE>(x, blk * B + (int64_t)(j * L + li) * CE, c);
      } else {
#pragma unroll
        for (int k = 0; k < CE; ++k) c[k] = 0.0f;
      }
#pragma unroll
      for (int k = 0; k < CE; ++k) v[t][j * CE + k] = c[k];
    }
  }
  prio_compute<ZQ_PRIO_QUANT>();
  const bool full = wg_blk0 + WG_BLOCKS <= nfull;  // workgroup-uniform
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int slot = t * WAVES + wave;              // tile index within the workgroup
    const int64_t blk = wg_blk0 + slot * BPW + lane / L;
    float a = fabsf(v[t][0]);
#pragma unroll
    for (int k = 1; k < E; ++k) a = fmaxf(a, fabsf(v[t][k]));
    const float amax = u2f(group_max<L>(f2u(a)));
    float s = 0.0f, r = 0.0f;
    if (amax >= kFlushBelow) {
      s = scale_of<(int)QMAX>(amax);
      r = QMAX / amax;
    }
    uint32_t m[E];
#pragma unroll
    for (int k = 0; k < E; ++k) m[k] = code_bits(v[t][k], r);

    // this lane's packed codes: OB bytes in element order (chunk j's codes are
    // bytes [j*OBC, (j+1)*OBC)), little-endian in w
    uint32_t w[NWO];
    if constexpr (QBITS == 8) {
#pragma unroll
      for (int k = 0; k < E / 4; ++k) w[k] = pack_bytes4(m[4 * k], m[4 * k + 1], m[4 * k + 2], m[4 * k + 3]);
    } else if constexpr (E == 4) {
      w[0] = (m[0] & 0xfu) | ((m[1] & 0xfu) << 4) | ((m[2] & 0xfu) << 8) | ((m[3] & 0xfu) << 12);
    } else {
#pragma unroll
      for (int k = 0; k < E / 8; ++k) w[k] = pack_nibbles8(m + 8 * k);
    }

    // chunk j's codes go to byte (j*L + li)*OBC of the block's codes
    if (full) {
      char* ob = reinterpret_cast<char*>(obuf) + (slot * BPW + lane / L) * BB;
#pragma unroll
      for (int j = 0; j < C; ++j) {
        char* d = ob + (j * L + li) * OBC;
        if constexpr (OBC == 2) {
          *reinterpret_cast<uint16_t*>(d) = (uint16_t)(w[j / 2] >> (16 * (j % 2)));
        } else {
#pragma unroll
          for (int k = 0; k < OBC / 4; ++k) reinterpret_cast<uint32_t*>(d)[k] = w[j * (OBC / 4) + k];
        }
      }
      if (li == 0) sbuf[slot * BPW + lane / L] = s;
    } else if (blk < nfull) {
      uint8_t* ob = out + blk * BB;
#pragma unroll
      for (int j = 0; j < C; ++j) {
        uint8_t* d = ob + (j * L + li) * OBC;
        if constexpr (OBC == 2) {
          st<NT>(reinterpret_cast<uint16_t*>(d), (uint16_t)(w[j / 2] >> (16 * (j % 2))));
        } else {
          uint32_t wc[OBC / 4];
#pragma unroll
          for (int k = 0; k < OBC / 4; ++k) wc[k] = w[j * (OBC / 4) + k];
          store_words<NT, OBC / 4>(d, wc);
        }
      }
      if (li == 0) st<2 * ZQ_NT_SCALES>(scales + blk, s);
    }
  }
  if (full) {
    __syncthreads();
    u32x4* dst = reinterpret_cast<u32x4*>(out + wg_blk0 * BB);
#pragma unroll
    for (int c = tid; c < WG_BYTES / 16; c += kQuantThreads) st<NT>(dst + c, obuf[c]);
    if (tid < WG_BLOCKS) st<2 * ZQ_NT_SCALES>(scales + wg_blk0 + tid, sbuf[tid]);
  }
}

// ------------------------------------------------------------------ dequantise
// INT8 (QBITS 8) or INT4 (QBITS 4) codes -> binary32 products -> DT.  Thread g
// < n/E owns elements [gE, gE + E) (one block, since E <= B); the n % E
// leftover elements go to the following threads, one each.  When a thread's
// output is wider than 16 bytes, a workgroup stages its outputs in LDS and
// writes them back as wave-contiguous 16-byte stores (wide per-lane writes
// lose bandwidth); the workgroup holding the end of the tensor stores
// directly.

template <int DT, int QBITS>
__global__ void __launch_bounds__(kDeqThreads) k_dequant(const uint8_t* __restrict__ codes,
                                                      const float* __restrict__ scales, int64_t n, int lgB,
                                                      void* __restrict__ y) {
  constexpr int E = QBITS == 8 ? deq8_elems(elem_size<DT>()) : deq4_elems(elem_size<DT>());
  constexpr int NT = QBITS == 8 ? ZQ_NT_DEQ8 : ZQ_NT_DEQ4;
  constexpr int IB = QBITS == 8 ? E : E / 2;  // code bytes per thread
  constexpr int OB = E * elem_size<DT>();     // output bytes per thread
  constexpr bool STAGE = ZQ_DEQ_STAGE && OB > 16;
  static_assert(IB % 4 == 0 && OB % 16 == 0, "lane layout");
  __shared__ u32x4 ybuf[STAGE ? kDeqThreads * OB / 16 : 1];

  const int64_t ngroups = n / E;
  const int64_t g0 = (int64_t)blockIdx.x * kDeqThreads;
  const int64_t gid = g0 + threadIdx.x;
  if (STAGE && g0 + kDeqThreads <= ngroups) {  // workgroup-uniform
    const int64_t e0 = gid * E;
    uint32_t w[IB / 4];
    prio_issue<ZQ_PRIO_DEQ>();
    load_words<NT, IB / 4>(codes + (e0 * IB) / E, w);
    const float s = ld<NT>(scales + (e0 >> lgB));
    prio_compute<ZQ_PRIO_DEQ>();
    float v[E];
#pragma unroll
    for (int k = 0; k < E; ++k) {
      if constexpr (QBITS == 8) v[k] = (float)(int32_t)(int8_t)(w[k >> 2] >> (8 * (k & 3))) * s;
      else v[k] = nib_to_f32(w[k >> 3], k & 7) * s;
    }
    store_elems<0, DT, E>(reinterpret_cast<char*>(ybuf) + threadIdx.x * OB, 0, v);
    __syncthreads();
    u32x4* dst = reinterpret_cast<u32x4*>(static_cast<char*>(y) + g0 * OB);
#pragma unroll
    for (int c = 0; c < OB / 16; ++c) st<NT>(dst + c * kDeqThreads + threadIdx.x, ybuf[c * kDeqThreads + threadIdx.x]);
  } else if (gid < ngroups) {
    const int64_t e0 = gid * E;
    uint32_t w[IB / 4];
    prio_issue<ZQ_PRIO_DEQ>();
    load_words<NT, IB / 4>(codes + (e0 * IB) / E, w);
    const float s = ld<NT>(scales + (e0 >> lgB));
    prio_compute<ZQ_PRIO_DEQ>();
    float v[E];
#pragma unroll
    for (int k = 0; k < E; ++k) {
      if constexpr (QBITS == 8) v[k] = (float)(int32_t)(int8_t)(w[k >> 2] >> (8 * (k & 3))) * s;
      else v[k] = nib_to_f32(w[k >> 3], k & 7) * s;
    }
    store_elems<NT, DT, E>(y, e0, v);
  } else if (gid - ngroups < n - ngroups * E) {
    const int64_t i = ngroups * E + (gid - ngroups);
    float prod;
    if constexpr (QBITS == 8) prod = (float)(int32_t)(int8_t)codes[i] * scales[i >> lgB];
    else prod = nib_to_f32(codes[i >> 1], (int)(i & 1)) * scales[i >> lgB];
    store1<DT>(y, i, prod);
  }
}

// ------------------------------------------------------------------ reduce level
// Vector path: slices 16-byte aligned (m % 32 == 0), blocks [0, nfull) with
// nfull a multiple of the group size GB below.  A lane owns E consecutive
// elements (E/2 bytes of every slice: consecutive lanes read consecutive
// bytes); L = B/E lanes hold one block; a wave tile is 64 lanes = BPW blocks.
// The 4 waves of a workgroup take 4 adjacent tiles (a group of GB blocks) and
// workgroup g processes groups g*TR .. g*TR + TR - 1.  Every load and store is
// addressed from a wave-uniform base plus the lane's offset, with no
// predicates.  Large levels use E = 32 (16 B per slice per lane), small levels
// (few waves, often many slices) E = 8, so that four times as many waves run.
//
// Slices are loaded U at a time (a batch).  With PIPE the batches of a
// workgroup's groups form one sequence of jobs whose register buffers
// alternate, so the loads of the next batch -- of this tile or of the next
// group -- are in flight while the current one is summed or the tile
// requantised; without it each batch is loaded, then summed.
//
// Per slice and element: one v_cvt_off_f32_i4 (q/16), one multiply by 16*s
// ((q/16)*(16 s) is the exact real q*s, so the rounded product is fl(q*s)),
// one add.  16*s is exact unless it overflows (s > 2^123, i.e. inputs above
// ~7e37); a wave holding such a scale multiplies by 16 first instead.  The
// first slice initialises the sum with its product: +0 + x = x for every x
// but -0, and a -0 sum and a +0 sum requantise to the same code and scale.
// Slices are summed in ascending order, exactly as defined.
//
// YDT >= 0 adds the fused final dequantisation: the requantised codes are
// turned back into fl(code * s_out) in YDT (the value qgz_dequantize would
// produce from this level's output) and written to y; out / sout may then be
// null, in which case the INT4 result is not stored.  Outputs wider than 16
// bytes per lane are staged in LDS and written as workgroup-contiguous
// 16-byte stores, as in the dequantiser.

// One slice into a lane's sum: acc[k] = fl(acc[k] + fl(q_k * s)) for the E
// codes of the NW words ww (FIRST: acc[k] = fl(q_k * s)).
template <int E, int NW, bool FIRST>
__device__ __forceinline__ void add_slice(float (&acc)[E], const uint32_t (&ww)[NW], float sc) {
  const float s16 = sc * 16.0f;
  if (__all(s16 <= kMaxFloat)) {  // wave-uniform: 16*s exact for every lane
#pragma unroll
    for (int j = 0; j < NW; ++j) {
      float f[8];
      nibbles_over_16(ww[j], f);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float prod = f[k] * s16;
        acc[8 * j + k] = FIRST ? prod : acc[8 * j + k] + prod;
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < NW; ++j) {
      float f[8];
      nibbles_over_16(ww[j], f);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float prod = (f[k] * 16.0f) * sc;
        acc[8 * j + k] = FIRST ? prod : acc[8 * j + k] + prod;
      }
    }
  }
}

// Requantise one wave tile (blocks from blk0, group grp) and store its INT4
// codes and scales (when out is not null) and, for YDT >= 0, the fused
// dequantisation fl(code * s_out) in YDT.  ybuf: the workgroup's LDS staging
// buffer for dequantised outputs wider than 16 bytes per lane; then every
// wave of the workgroup must call this for the same group.
template <int B, int E, int YDT>
__device__ __forceinline__ void requant_tile(const float (&acc)[E], int64_t blk0, int64_t grp, int lane,
                                             uint8_t* __restrict__ out, float* __restrict__ sout,
                                             void* __restrict__ y, u32x4* ybuf) {
  constexpr int L = B / E, NW = E / 8, GB = kThreads / 64 * (64 / L);
  constexpr int YB = YDT < 0 ? 0 : E * elem_size<(YDT < 0 ? 0 : YDT)>();  // dequantised bytes per lane
  float a = fabsf(acc[0]);
#pragma unroll
  for (int k = 1; k < E; ++k) a = fmaxf(a, fabsf(acc[k]));
  const float amax = u2f(group_max<L>(f2u(a)));
  float so = 0.0f, r = 0.0f;
  if (amax >= kFlushBelow) {
    so = scale_of<7>(amax);
    r = 7.0f / amax;
  }
  uint32_t m[E];
#pragma unroll
  for (int k = 0; k < E; ++k) m[k] = code_bits(acc[k], r);
  if (out != nullptr) {
    uint32_t o[NW];
#pragma unroll
    for (int j = 0; j < NW; ++j) o[j] = pack_nibbles8(m + 8 * j);
    store_words<ZQ_NT_REDUCE, NW>(out + blk0 * (B / 2) + lane * (E / 2), o);
    if (lane % L == 0) st<2 * ZQ_NT_SCALES>(sout + blk0 + lane / L, so);
  }
  if constexpr (YDT >= 0) {
    // code as float: (1.5*2^23 + q) - 1.5*2^23 = q exactly; then fl(q * s_out)
    float v[E];
#pragma unroll
    for (int k = 0; k < E; ++k) v[k] = (u2f(m[k]) - kRoundMagic) * so;
    if constexpr (YB > 16) {  // every wave of the workgroup is here, at the same group
      store_elems<0, YDT, E>(reinterpret_cast<char*>(ybuf) + threadIdx.x * YB, 0, v);
      __syncthreads();
      u32x4* dst = reinterpret_cast<u32x4*>(static_cast<char*>(y) + grp * GB * B * elem_size<YDT>());
#pragma unroll
      for (int c = 0; c < YB / 16; ++c)
        st<ZQ_NT_DEQ4>(dst + c * kThreads + threadIdx.x, ybuf[c * kThreads + threadIdx.x]);
      __syncthreads();
    } else {
      store_elems<ZQ_NT_DEQ4, YDT, E>(y, blk0 * B + (int64_t)lane * E, v);
    }
  }
}

template <int U, int NW>
struct SliceBatch {
  uint32_t w[U][NW];
  float s[U];
};

// GATHER: the slices are not back to back; `in` and `sin` point to device
// tables of P slice pointers (bytes, scales) instead, e.g. the peers' send
// buffers mapped into this GPU's address space.
template <int B, int E, int U, int TR, bool PIPE, int YDT, bool GATHER = false>
__global__ void __launch_bounds__(kThreads) k_reduce(const uint8_t* __restrict__ in, const float* __restrict__ sin,
                                                     int P, int64_t slice_bytes, int64_t slice_scales,
                                                     int64_t nfull, uint8_t* __restrict__ out,
                                                     float* __restrict__ sout, void* __restrict__ y) {
  constexpr int L = B / E, BPW = 64 / L, NW = E / 8, WPG = kThreads / 64, GB = WPG * BPW;
  static_assert(L >= 1 && L <= 64 && (NW == 1 || NW == 2 || NW == 4) && TR >= 1, "lane layout");
  constexpr int YB = YDT < 0 ? 0 : E * elem_size<(YDT < 0 ? 0 : YDT)>();  // dequantised bytes per lane
  constexpr bool YSTAGE = YB > 16;
  __shared__ u32x4 ybuf[YSTAGE ? kThreads * YB / 16 : 1];
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane_byte = lane * (E / 2);

  const int64_t g0 = (int64_t)blockIdx.x * TR;  // first group of this workgroup
  const int64_t groups = nfull / GB;
  const int ng = (int)(groups - g0 >= TR ? TR : groups - g0);  // >= 1 by the launch size
  const int nb = (P + U - 1) / U;
  auto tile_blk0 = [&](int64_t grp) { return (grp * WPG + wv) * BPW; };

  // slices [b*U, b*U + U) of this wave's tile of group grp
  auto issue = [&](SliceBatch<U, NW>& X, int64_t grp, int b) {
    const int64_t blk0 = tile_blk0(grp);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int p = b * U + u;
      if (p < P) {
        const uint8_t* tb;
        const float* sb;
        if constexpr (GATHER) {
          tb = reinterpret_cast<const uint8_t* const*>(in)[p] + blk0 * (B / 2);
          sb = reinterpret_cast<const float* const*>(sin)[p] + blk0;
        } else {
          tb = in + blk0 * (B / 2) + (int64_t)p * slice_bytes;
          sb = sin + blk0 + (int64_t)p * slice_scales;
        }
        load_words<ZQ_NT_REDUCE, NW>(tb + lane_byte, X.w[u]);
        X.s[u] = ld<ZQ_NT_REDUCE>(sb + lane / L);
      }
    }
  };

  float acc[E];
  auto sum_batch = [&](const SliceBatch<U, NW>& X, int b) {
    if (b == 0) add_slice<E, NW, true>(acc, X.w[0], X.s[0]);
    else add_slice<E, NW, false>(acc, X.w[0], X.s[0]);
#pragma unroll
    for (int u = 1; u < U; ++u)
      if (b * U + u < P) add_slice<E, NW, false>(acc, X.w[u], X.s[u]);
  };
  // requantise this wave's tile of group grp and store it
  auto finish = [&](int64_t grp) { requant_tile<B, E, YDT>(acc, tile_blk0(grp), grp, lane, out, sout, y, ybuf); };

  SliceBatch<U, NW> A;
  if constexpr (!PIPE) {
#pragma unroll 1
    for (int t = 0; t < ng; ++t) {
#pragma unroll 1
      for (int b = 0; b < nb; ++b) {
        issue(A, g0 + t, b);
        sum_batch(A, b);
      }
      finish(g0 + t);
    }
  } else {
    // jobs (group g0 + t, batch b) in order, two buffers alternating
    SliceBatch<U, NW> Bf;
    const int njobs = ng * nb;
    int it = 0, ib = 0, ct = 0, cb = 0;  // next job to issue / to consume
    auto next = [&](int& t, int& b) {
      if (++b == nb) {
        b = 0;
        ++t;
      }
    };
    issue(A, g0 + it, ib);
    next(it, ib);
#pragma unroll 1
    for (int j = 0; j < njobs; j += 2) {
      if (j + 1 < njobs) {
        issue(Bf, g0 + it, ib);
        next(it, ib);
      }
      sum_batch(A, cb);
      if (cb == nb - 1) finish(g0 + ct);
      next(ct, cb);
      if (j + 2 < njobs) {
        issue(A, g0 + it, ib);
        next(it, ib);
      }
      if (j + 1 < njobs) {
        sum_batch(Bf, cb);
        if (cb == nb - 1) finish(g0 + ct);
        next(ct, cb);
      }
    }
  }
}

// Vector path with the slice count fixed at compile time (PC = 2, 4 or 8;
// E = 32 on large levels, E = 8 on small ones).  Same lane layout,
// arithmetic and order as k_reduce, but every load is
// unconditional, so the compiler waits for each slice's data on its own
// (s_waitcnt vmcnt(n) counting the loads issued after it) instead of for
// every load in flight, and the sum of slice 0 starts while the others are
// still arriving.  A workgroup takes TRC consecutive groups; with TRC > 1 the
// loads of a wave's next tile are issued before its current tile is summed,
// so they arrive while it computes (two register buffers).  The last
// workgroup clamps its group index to the last group and recomputes it,
// rewriting identical values, instead of branching around loads.
#ifndef ZQ_FIXED_WAVES
#define ZQ_FIXED_WAVES 0
#endif
#if ZQ_FIXED_WAVES
#define ZQ_FIXED_ATTR __attribute__((amdgpu_waves_per_eu(ZQ_FIXED_WAVES)))
#else
#define ZQ_FIXED_ATTR
#endif
template <int B, int E, int PC, int TRC, int YDT, bool GATHER>
__global__ void __launch_bounds__(kThreads) ZQ_FIXED_ATTR k_reduce_p(const uint8_t* __restrict__ in, const float* __restrict__ sin,
                                                       int, int64_t slice_bytes, int64_t slice_scales, int64_t nfull,
                                                       uint8_t* __restrict__ out, float* __restrict__ sout,
                                                       void* __restrict__ y) {
  constexpr int L = B / E, BPW = 64 / L, NW = E / 8, WPG = kThreads / 64, GB = WPG * BPW, NBUF = TRC > 1 ? 2 : 1;
  static_assert(L >= 1 && L <= 64 && (NW == 1 || NW == 2 || NW == 4) && PC >= 1 && TRC >= 1, "lane layout");
  constexpr int YB = YDT < 0 ? 0 : E * elem_size<(YDT < 0 ? 0 : YDT)>();
  __shared__ u32x4 ybuf[YB > 16 ? kThreads * YB / 16 : 1];
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane_byte = lane * (E / 2);
  const int64_t last = nfull / GB - 1;                  // last group
  const int64_t g0 = (int64_t)blockIdx.x * TRC;
  auto group_of = [&](int t) { return g0 + t < last ? g0 + t : last; };
  auto tile_blk0 = [&](int64_t grp) { return (grp * WPG + wv) * BPW; };

  uint32_t w[NBUF][PC][NW];
  float sc[NBUF][PC];
  auto issue = [&](int buf, int64_t grp) {
    const int64_t blk0 = tile_blk0(grp);
#pragma unroll
    for (int p = 0; p < PC; ++p) {
      const uint8_t* tb;
      const float* sb;
      if constexpr (GATHER) {
        tb = reinterpret_cast<const uint8_t* const*>(in)[p] + blk0 * (B / 2);
        sb = reinterpret_cast<const float* const*>(sin)[p] + blk0;
      } else {
        tb = in + blk0 * (B / 2) + (int64_t)p * slice_bytes;
        sb = sin + blk0 + (int64_t)p * slice_scales;
      }
      load_words<ZQ_NT_REDUCE, NW>(tb + lane_byte, w[buf][p]);
      sc[buf][p] = ld<ZQ_NT_REDUCE>(sb + lane / L);
    }
  };

  prio_issue<ZQ_PRIO_REDUCE>();
  issue(0, group_of(0));
  prio_compute<ZQ_PRIO_REDUCE>();
#pragma unroll
  for (int t = 0; t < TRC; ++t) {
    if (t + 1 < TRC) {
      prio_issue<ZQ_PRIO_REDUCE>();
      issue((t + 1) % NBUF, group_of(t + 1));
      prio_compute<ZQ_PRIO_REDUCE>();
    }
    const int b = t % NBUF;
    float acc[E];
    add_slice<E, NW, true>(acc, w[b][0], sc[b][0]);
#pragma unroll
    for (int p = 1; p < PC; ++p) add_slice<E, NW, false>(acc, w[b][p], sc[b][p]);
    const int64_t grp = group_of(t);
    requant_tile<B, E, YDT>(acc, tile_blk0(grp), grp, lane, out, sout, y, ybuf);
  }
}

// Generic path: any m, any slice alignment; one wave per block, blocks
// [blk_begin, blk_begin + gridDim.x).  A lane owns byte j = lane + 64 i of the
// block (elements 2j, 2j+1), i < B/128 rounded up.  Plain arithmetic, the
// definition as written: sum from +0, one multiply and one add per slice.
// GATHER as for k_reduce.
template <bool GATHER>
__global__ void __launch_bounds__(64) k_reduce_generic(const uint8_t* __restrict__ in, const float* __restrict__ sin,
                                                       int P, int64_t slice_bytes, int64_t slice_scales, int64_t m,
                                                       int B, int64_t blk_begin, uint8_t* __restrict__ out,
                                                       float* __restrict__ sout, void* __restrict__ y, int ydt) {
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
    const float s = GATHER ? reinterpret_cast<const float* const*>(sin)[p][blk] : sin[(int64_t)p * slice_scales + blk];
    const uint8_t* src =
        (GATHER ? reinterpret_cast<const uint8_t* const*>(in)[p] : in + (int64_t)p * slice_bytes) + (base >> 1);
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
    so = scale_of<7>(amax);
    r = 7.0f / amax;
  }
#pragma unroll
  for (int i = 0; i < MAXI; ++i) {
    const int j = lane + 64 * i;
    if (j < nbytes) {
      const uint32_t lo = code_bits(acc[2 * i], r);
      const uint32_t hi = (2 * j + 1 < len) ? code_bits(acc[2 * i + 1], r) : 0u;
      if (out != nullptr) out[(base >> 1) + j] = (uint8_t)((lo & 0xfu) | ((hi & 0xfu) << 4));
      if (y != nullptr) {
        const float v0 = (u2f(lo) - kRoundMagic) * so, v1 = (u2f(hi) - kRoundMagic) * so;
        const int64_t i0 = base + 2 * j;
        if (ydt == ZQ_F32) store1<ZQ_F32>(y, i0, v0);
        else if (ydt == ZQ_F16) store1<ZQ_F16>(y, i0, v0);
        else store1<ZQ_BF16>(y, i0, v0);
        if (2 * j + 1 < len) {
          if (ydt == ZQ_F32) store1<ZQ_F32>(y, i0 + 1, v1);
          else if (ydt == ZQ_F16) store1<ZQ_F16>(y, i0 + 1, v1);
          else store1<ZQ_BF16>(y, i0 + 1, v1);
        }
      }
    }
  }
  if (lane == 0 && out != nullptr) sout[blk] = so;
}

// ------------------------------------------------------------------ address tables
// Writes count (<= kTableChunk) 64-bit entries carried in the kernel
// arguments to dst[0, count): lane t stores entry t with a vector store.
__global__ void __launch_bounds__(kTableChunk) k_fill_table(uint64_t* __restrict__ dst, TableChunk chunk, int count) {
  const int t = threadIdx.x;
  if (t < count) dst[t] = chunk.v[t];
}

FillTableKernel fill_table_kernel() { return &k_fill_table; }

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

DequantKernel dequant_kernel(int dt, int qbits) {
  if (qbits == 8) {
    if (dt == ZQ_F32) return &k_dequant<ZQ_F32, 8>;
    if (dt == ZQ_F16) return &k_dequant<ZQ_F16, 8>;
    return &k_dequant<ZQ_BF16, 8>;
  }
  if (dt == ZQ_F32) return &k_dequant<ZQ_F32, 4>;
  if (dt == ZQ_F16) return &k_dequant<ZQ_F16, 4>;
  return &k_dequant<ZQ_BF16, 4>;
}

template <int YDT>
static ReduceKernel reduce_kernel_for(int lgB, ReduceShape shape) {
  // large: E = 32, U = 4; two slices: E = 32, U = 2, two tiles per wave with the
  // next tile's loads issued before this tile's requantisation; small: E = 8,
  // U = 16.  A block may span at most one wave, so B = 1024 always takes large.
  constexpr int EL = kReduceElems, UL = ZQ_REDUCE_U, ES = kReduceElemsSmall, US = ZQ_REDUCE_U_SMALL;
  constexpr int TL = reduce_tiles(ReduceShape::kLarge), T2 = reduce_tiles(ReduceShape::kTwoSlices),
                TS = reduce_tiles(ReduceShape::kSmall);
  constexpr bool PL = ZQ_REDUCE_PIPE, P2 = ZQ_REDUCE_PIPE2, PS = ZQ_REDUCE_PIPE_SMALL;
#define ZQ_REDUCE_CASE(LG, BB)                                                                       \
  case LG:                                                                                           \
    if (shape == ReduceShape::kSmall) return &k_reduce<BB, ES, US, TS, PS, YDT>;                     \
    if (shape == ReduceShape::kTwoSlices) return &k_reduce<BB, EL, 2, T2, P2, YDT>;                  \
    return &k_reduce<BB, EL, UL, TL, PL, YDT>;
  switch (lgB) {
    ZQ_REDUCE_CASE(5, 32)
    ZQ_REDUCE_CASE(6, 64)
    ZQ_REDUCE_CASE(7, 128)
    ZQ_REDUCE_CASE(8, 256)
    ZQ_REDUCE_CASE(9, 512)
    default: return &k_reduce<1024, EL, UL, TL, PL, YDT>;
  }
#undef ZQ_REDUCE_CASE
}

ReduceKernel reduce_kernel(int lgB, ReduceShape shape, int ydt) {
  switch (ydt) {
    case ZQ_F32: return reduce_kernel_for<ZQ_F32>(lgB, shape);
    case ZQ_F16: return reduce_kernel_for<ZQ_F16>(lgB, shape);
    case ZQ_BF16: return reduce_kernel_for<ZQ_BF16>(lgB, shape);
    default: return reduce_kernel_for<-1>(lgB, shape);
  }
}

ReduceKernel reduce_gather_kernel(int lgB, ReduceShape shape) {
  constexpr int EL = kReduceElems, UL = ZQ_REDUCE_U, ES = kReduceElemsSmall, US = ZQ_REDUCE_U_SMALL;
  constexpr int TL = reduce_tiles(ReduceShape::kLarge), T2 = reduce_tiles(ReduceShape::kTwoSlices),
                TS = reduce_tiles(ReduceShape::kSmall);
  constexpr bool PL = ZQ_REDUCE_PIPE, P2 = ZQ_REDUCE_PIPE2, PS = ZQ_REDUCE_PIPE_SMALL;
#define ZQ_GATHER_CASE(LG, BB)                                                                        \
  case LG:                                                                                            \
    if (shape == ReduceShape::kSmall) return &k_reduce<BB, ES, US, TS, PS, -1, true>;                 \
    if (shape == ReduceShape::kTwoSlices) return &k_reduce<BB, EL, 2, T2, P2, -1, true>;              \
    return &k_reduce<BB, EL, UL, TL, PL, -1, true>;
  switch (lgB) {
    ZQ_GATHER_CASE(5, 32)
    ZQ_GATHER_CASE(6, 64)
    ZQ_GATHER_CASE(7, 128)
    ZQ_GATHER_CASE(8, 256)
    ZQ_GATHER_CASE(9, 512)
    default: return &k_reduce<1024, EL, UL, TL, PL, -1, true>;
  }
#undef ZQ_GATHER_CASE
}

#ifndef ZQ_FIXED_TR2
#define ZQ_FIXED_TR2 4
#endif
#ifndef ZQ_FIXED_TR4
#define ZQ_FIXED_TR4 1
#endif
#ifndef ZQ_FIXED_TR8
#define ZQ_FIXED_TR8 1
#endif
constexpr int fixed_tiles(int P) { return P == 2 ? ZQ_FIXED_TR2 : P == 4 ? ZQ_FIXED_TR4 : ZQ_FIXED_TR8; }
int reduce_fixed_tiles(int P) { return fixed_tiles(P); }

#ifndef ZQ_FIXED_E
#define ZQ_FIXED_E 32
#endif
#ifndef ZQ_FIXED_SMALL
#define ZQ_FIXED_SMALL 1
#endif
int reduce_fixed_elems() { return ZQ_FIXED_E; }

template <int B, int YDT, bool GATHER>
static ReduceKernel reduce_fixed_for_b(int P) {
  constexpr int E = ZQ_FIXED_E;
  if (P == 2) return &k_reduce_p<B, E, 2, fixed_tiles(2), YDT, GATHER>;
  if (P == 4) return &k_reduce_p<B, E, 4, fixed_tiles(4), YDT, GATHER>;
  return &k_reduce_p<B, E, 8, fixed_tiles(8), YDT, GATHER>;
}

template <int YDT, bool GATHER>
static ReduceKernel reduce_fixed_for(int lgB, int P) {
  if (lgB == 6) return reduce_fixed_for_b<64, YDT, GATHER>(P);
  if (lgB == 7) return reduce_fixed_for_b<128, YDT, GATHER>(P);
  return reduce_fixed_for_b<256, YDT, GATHER>(P);
}

ReduceKernel reduce_fixed_kernel(int lgB, int P, int ydt, bool gather) {
  if (lgB < 6 || lgB > 8 || (P != 2 && P != 4 && P != 8) || (gather && ydt >= 0)) return nullptr;
  if (gather) return reduce_fixed_for<-1, true>(lgB, P);
  switch (ydt) {
    case ZQ_F32: return reduce_fixed_for<ZQ_F32, false>(lgB, P);
    case ZQ_F16: return reduce_fixed_for<ZQ_F16, false>(lgB, P);
    case ZQ_BF16: return reduce_fixed_for<ZQ_BF16, false>(lgB, P);
    default: return reduce_fixed_for<-1, false>(lgB, P);
  }
}

// Small levels (E = 8, the small-level group size): P = 2, 4, 8 fixed at
// compile time, one group per workgroup.
template <int B, int YDT, bool GATHER>
static ReduceKernel reduce_fixed_small_for_b(int P) {
  if (P == 2) return &k_reduce_p<B, 8, 2, 1, YDT, GATHER>;
  if (P == 4) return &k_reduce_p<B, 8, 4, 1, YDT, GATHER>;
  return &k_reduce_p<B, 8, 8, 1, YDT, GATHER>;
}

template <int YDT, bool GATHER>
static ReduceKernel reduce_fixed_small_for(int lgB, int P) {
  if (lgB == 6) return reduce_fixed_small_for_b<64, YDT, GATHER>(P);
  if (lgB == 7) return reduce_fixed_small_for_b<128, YDT, GATHER>(P);
  return reduce_fixed_small_for_b<256, YDT, GATHER>(P);
}

ReduceKernel reduce_fixed_small_kernel(int lgB, int P, int ydt, bool gather) {
  if (!ZQ_FIXED_SMALL || lgB < 6 || lgB > 8 || (P != 2 && P != 4 && P != 8) || (gather && ydt >= 0)) return nullptr;
  if (gather) return reduce_fixed_small_for<-1, true>(lgB, P);
  switch (ydt) {
    case ZQ_F32: return reduce_fixed_small_for<ZQ_F32, false>(lgB, P);
    case ZQ_F16: return reduce_fixed_small_for<ZQ_F16, false>(lgB, P);
    case ZQ_BF16: return reduce_fixed_small_for<ZQ_BF16, false>(lgB, P);
    default: return reduce_fixed_small_for<-1, false>(lgB, P);
  }
}

ReduceGenericKernel reduce_generic_kernel(bool gather) {
  return gather ? &k_reduce_generic<true> : &k_reduce_generic<false>;
}

}  // namespace zq
