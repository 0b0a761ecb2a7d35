// zq_gemm.hip -- dequantise-on-load GEMM for gfx950 MFMA.
//
// The gathered INT8 layer feeds the forward matmuls of that layer (the paper's
// Design, Weight Partitioning: the Allgathered weights are dequantised for the
// forward pass).  Instead of writing the dequantised bf16 / fp16 layer to HBM
// and reading it back in the matmul, this kernel dequantises each weight tile
// as it is staged into LDS:
//
//   y[m][n] = sum_k x[m][k] * w[n][k],   w[n][k] = cvt(fl(q[n*K + k] * s[(n*K + k) / B]))
//
// with q / s the qwZ codes and block scales of the N x K weight (PyTorch
// Linear layout, flat row-major) and cvt the nearest-even narrowing to x's
// type -- exactly the values qwz_dequantize writes.  Products are exact in
// binary32 and summed in binary32 by the MFMA units (v_mfma_f32_32x32x16_bf16
// / _f16), in an order the hardware fixes.
//
// Kernels:
//   k_dqgemv     M <= 16: weight streaming on 16 x 16 x 32 MFMAs, codes loaded
//                straight into the operand registers, x staged in LDS once
//                per K range (see the kernel).
//   k_dqgemm_pp  M > 16: 256 x 256 tiles (128 x 256 up to 128 rows) over 8
//                waves in a ping-pong schedule, waves w and w + 4 of a SIMD
//                half a K-step apart (one stores the next tile and reads its
//                fragments while the other runs its MFMAs, with its loads
//                and dequantisation in between); buffer loads, none
//                predicated; K split across workgroups where the tiles are
//                too few to fill the GPU.
//   k_dqgemm     the same 256 x 256 tiles in a plain two-stage schedule with
//                64-bit addresses, for K > kDqGemmPpMaxK.
// The tiled kernels use 32 x 32 MFMA tiles, K advancing 64 at a time, LDS
// rows padded by 16 bytes so that the 16-byte fragment reads of 16
// consecutive lanes fall in distinct banks.
// Many-row workgroups are numbered so that each XCD receives a contiguous
// range of tiles, and within it groups of 4 tile rows share their weight
// tiles through that XCD's L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "zq.h"
#include "zq_device.h"
#include "zq_host.h"

#pragma clang fp contract(off)

namespace zq {

// dequantise-on-load GEMM (x of type xt = ZQ_BF16 or ZQ_F16)
#ifndef ZQ_GEMM_BM
#define ZQ_GEMM_BM 256
#endif
#ifndef ZQ_GEMM_BN
#define ZQ_GEMM_BN 256
#endif
#ifndef ZQ_GEMM_WM
#define ZQ_GEMM_WM 2
#endif
#ifndef ZQ_GEMM_WN
#define ZQ_GEMM_WN 4
#endif
#ifndef ZQ_GEMM_PINGPONG
#define ZQ_GEMM_PINGPONG 1
#endif
constexpr int kDqGemmTileM = ZQ_GEMM_BM;  // rows of y per workgroup
constexpr int kDqGemmTileN = ZQ_GEMM_BN;  // columns of y per workgroup
constexpr int kDqGemmK = 64;              // K must be a multiple of this
constexpr int kDqGemmThreads = 64 * ZQ_GEMM_WM * ZQ_GEMM_WN;
constexpr int64_t kDqGemmPpMaxK = int64_t(1) << 21;  // 32-bit buffer offsets in the ping-pong kernel
// K splits of the ping-pong kernel when its tiles leave CUs idle
#ifndef ZQ_GEMM_PP_MAX_SPLITS
#define ZQ_GEMM_PP_MAX_SPLITS 16
#endif
// the split model's two costs: one 64-wide K-step of a 256 x 256 tile on one
// CU, and one atomic addition into y with the GPU's others (measured: a K-step
// 1.3-1.7 us, atomic additions about 330 G/s)
#ifndef ZQ_GEMM_PP_STEP_NS
#define ZQ_GEMM_PP_STEP_NS 1500
#endif
#ifndef ZQ_GEMM_ATOMIC_PS
#define ZQ_GEMM_ATOMIC_PS 3
#endif
constexpr int64_t kDqGemmMaxSplits = ZQ_GEMM_PP_MAX_SPLITS;
// Row ranges: M <= 16 the weight-streaming kernel k_dqgemv; up to
// ZQ_GEMM_HALF_M rows the ping-pong kernel's 128 x 256 tiles; beyond, its
// 256 x 256 tiles.  Measured over the layer's four GEMMs in sequence: the
// streaming kernel 0.11-0.15 ms at 1-16 tokens against 0.17 for the ping-pong
// kernel; the 128 x 256 tiles 10-14% faster than the 256 x 256 at 65-128
// rows and slower at 144-224; and both faster than a 64 x 64 few-row tile
// kernel (since removed) from 24 rows on.
#ifndef ZQ_GEMM_HALF_M
#define ZQ_GEMM_HALF_M 128
#endif
// the weight-streaming kernel aims at this many workgroups
#ifndef ZQ_GEMM_GEMV_TARGET
#define ZQ_GEMM_GEMV_TARGET 1024
#endif
constexpr int64_t kGemvTargetWgs = ZQ_GEMM_GEMV_TARGET;
using DqGemmKernel = void (*)(const uint16_t*, const int8_t*, const float*, int64_t, int64_t, int64_t, int, float*,
                              int64_t, int64_t, int);

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kBK = 64;
// buffer resource word 3 for raw (untyped) buffer loads on gfx9-family targets
constexpr int kBufferFlags = 0x00020000;
constexpr int kLDK = kBK + 8;  // LDS row stride in 16-bit elements (144 bytes)
constexpr int kRow16 = kLDK / 8;  // the same in 16-byte units
#ifndef ZQ_GEMM_GROUP_M
#define ZQ_GEMM_GROUP_M 4
#endif
#ifndef ZQ_GEMM_XCD_MAP
#define ZQ_GEMM_XCD_MAP 1
#endif
constexpr int kGroupM = ZQ_GEMM_GROUP_M;  // tile rows sharing a weight tile in L2
constexpr int kXcds = 8;

// f(integral_constant<int, i>) for i = I .. N - 1
template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

template <int XT>
__device__ __forceinline__ f32x16_t mfma32(u32x4 a, u32x4 b, f32x16_t c) {
  if constexpr (XT == ZQ_BF16)
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b), c,
                                                  0, 0, 0);
}

// two binary32 values narrowed to XT, packed low-first
template <int XT>
__device__ __forceinline__ uint32_t narrow2(float a, float b) {
  if constexpr (XT == ZQ_BF16) return bf16x2_bits(a, b);
  else return f2h(a) | (f2h(b) << 16);
}

// BM x BN tile of y per workgroup, WM x WN waves, each wave a (BM/WM) x (BN/WN)
// block of 32 x 32 MFMA tiles, with plain loads and 64-bit addresses (the
// schedule for K beyond the ping-pong kernel's 32-bit offsets); `splits` is
// unused (the launch signature is shared with k_dqgemm_pp).
template <int XT, int BM, int BN, int WM, int WN>
__global__ void __launch_bounds__(64 * WM * WN) k_dqgemm(const uint16_t* __restrict__ x, const int8_t* __restrict__ codes,
                                                         const float* __restrict__ scales, int64_t M, int64_t N,
                                                         int64_t K, int lgB, float* __restrict__ y, int64_t mtiles,
                                                         int64_t ntiles, int splits) {
  constexpr int NT = 64 * WM * WN;                         // threads
  constexpr int TI = BM / WM / 32, TJ = BN / WN / 32;      // MFMA tiles per wave
  constexpr int XC = BM * kBK / 8 / NT;                    // x chunks (8 elements) per thread
  constexpr int WC = BN * kBK / 16 / NT;                   // code chunks (16 codes) per thread
  static_assert(TI >= 1 && TJ >= 1 && XC >= 1 && WC >= 1 && XC * NT * 8 == BM * kBK && WC * NT * 16 == BN * kBK,
                "tile shape");
  __shared__ u32x4 As[2][BM * kLDK / 8];
  __shared__ u32x4 Bs[2][BN * kLDK / 8];

  // workgroup -> tile: XCD-contiguous ranges (workgroups are dealt to the
  // XCDs round robin), then column-major groups of kGroupM tile rows
  const int64_t T = mtiles * ntiles;
  const int64_t wg = blockIdx.x;
  const int64_t q = T / kXcds, r = T % kXcds, xcd = wg % kXcds, idx = wg / kXcds;
  const int64_t t = !ZQ_GEMM_XCD_MAP ? wg : xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
  const int64_t per_group = (int64_t)kGroupM * ntiles;
  const int64_t first_m = (t / per_group) * kGroupM;
  const int64_t gsize = mtiles - first_m < kGroupM ? mtiles - first_m : kGroupM;
  const int64_t mt = first_m + (t % per_group) % gsize;
  const int64_t nt = (t % per_group) / gsize;
  const int64_t m0 = mt * BM, n0 = nt * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, wm = wave / WN, wn = wave % WN;
  const int KT = (int)(K / kBK);
  (void)splits;

  // two register sets: tile t's loads are issued two K-steps before its LDS
  // store
  u32x4 xrs[2][XC], wrs[2][WC];
  float srs[2][WC];
  // global -> registers: x rows m0.., 8 elements per chunk; codes rows n0..,
  // 16 codes per chunk with the scale of their block (a chunk never straddles
  // a block: chunks are 16-aligned in the flat index and B >= 32)
  auto gload = [&](int kt, auto rs_c) {
    constexpr int R = decltype(rs_c)::value;
    u32x4(&xr)[XC] = xrs[R];
    u32x4(&wr)[WC] = wrs[R];
    float(&sr)[WC] = srs[R];
    const int64_t k0 = (int64_t)kt * kBK;
#pragma unroll
    for (int i = 0; i < XC; ++i) {
      const int c = tid + NT * i, row = c >> 3, col = (c & 7) * 8;
      const int64_t m = m0 + row;
      xr[i] = m < M ? *reinterpret_cast<const u32x4*>(x + m * K + k0 + col) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < WC; ++i) {
      const int c = tid + NT * i, row = c >> 2, col = (c & 3) * 16;
      const int64_t n = n0 + row;
      if (n < N) {
        const int64_t f = n * K + k0 + col;
        wr[i] = *reinterpret_cast<const u32x4*>(codes + f);
        sr[i] = scales[f >> lgB];
      } else {
        wr[i] = u32x4{0u, 0u, 0u, 0u};
        sr[i] = 0.0f;
      }
    }
  };
  // registers -> LDS buffer `buf`; codes become fl(q * s) narrowed to XT
  auto sstore = [&](int buf, auto rs_c) {
    constexpr int R = decltype(rs_c)::value;
    const u32x4(&xr)[XC] = xrs[R];
    const u32x4(&wr)[WC] = wrs[R];
    const float(&sr)[WC] = srs[R];
#pragma unroll
    for (int i = 0; i < XC; ++i) {
      const int c = tid + NT * i, row = c >> 3, col = (c & 7) * 8;
      As[buf][(row * kLDK + col) / 8] = xr[i];
    }
#pragma unroll
    for (int i = 0; i < WC; ++i) {
      const int c = tid + NT * i, row = c >> 2, col = (c & 3) * 16;
      uint32_t o[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t word = wr[i][j >> 1];
        const int sh = (j & 1) * 16;
        const float v0 = (float)(int32_t)(int8_t)(word >> sh) * sr[i];
        const float v1 = (float)(int32_t)(int8_t)(word >> (sh + 8)) * sr[i];
        o[j] = narrow2<XT>(v0, v1);
      }
      Bs[buf][(row * kLDK + col) / 8] = u32x4{o[0], o[1], o[2], o[3]};
      Bs[buf][(row * kLDK + col) / 8 + 1] = u32x4{o[4], o[5], o[6], o[7]};
    }
  };

  f32x16_t acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  // MFMA operands: lane l holds row (l % 32) of its 32-row tile, k elements
  // [8 (l / 32), 8 (l / 32) + 8) of the 16-wide step
  const int frow = lane & 31, fk = 8 * (lane >> 5);
  auto compute = [&](int buf) {
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      u32x4 a[TI], b[TJ];
#pragma unroll
      for (int i = 0; i < TI; ++i) a[i] = As[buf][((wm * TI * 32 + i * 32 + frow) * kLDK + kk * 16 + fk) / 8];
#pragma unroll
      for (int j = 0; j < TJ; ++j) b[j] = Bs[buf][((wn * TJ * 32 + j * 32 + frow) * kLDK + kk * 16 + fk) / 8];
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) acc[i][j] = mfma32<XT>(a[i], b[j], acc[i][j]);
    }
  };

  using R0 = std::integral_constant<int, 0>;
  using R1 = std::integral_constant<int, 1>;
  // tile t lives in register set t % 2 from its load (K-step t - 2) to its
  // store (end of K-step t - 1)
  if (KT > 0) {
    gload(0, R0{});
    sstore(0, R0{});
  }
  if (KT > 1) gload(1, R1{});
  if (KT > 2) gload(2, R0{});
  __syncthreads();
#pragma unroll 1
  for (int kt = 0; kt < KT; kt += 2) {
    compute(0);                                   // K-step kt (buffer 0)
    if (kt + 1 < KT) sstore(1, R1{});             // tile kt + 1
    if (kt + 3 < KT) gload(kt + 3, R1{});
    __syncthreads();
    if (kt + 1 < KT) {
      compute(1);                                 // K-step kt + 1 (buffer 1)
      if (kt + 2 < KT) sstore(0, R0{});           // tile kt + 2
      if (kt + 4 < KT) gload(kt + 4, R0{});
      __syncthreads();
    }
  }

  // D register e of lane l: row 8 (e / 4) + 4 (l / 32) + e % 4, column l % 32
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int64_t n = n0 + wn * TJ * 32 + j * 32 + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t m = m0 + wm * TI * 32 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (m < M && n < N) y[m * N + n] = acc[i][j][e];
      }
    }
}

// The 256 x 256 tile with a ping-pong schedule (8 waves, two per SIMD).  Waves
// w and w + 4 share a SIMD (a workgroup's waves are dealt to the 4 SIMDs round
// robin) and run half a K-step (32 of K) out of phase: while one runs the 16
// MFMAs of its half (with its next global loads and the dequantisation of its
// next weight chunk interleaved), the other stores its part of the next tile
// into LDS and reads its next operand fragments, so the matrix core of each
// SIMD stays fed.  Each phase ends in a
// workgroup barrier, which also orders the LDS traffic: tile kt + 1 is written
// during the four phases of K-step kt (two per wave group) into the buffer
// that tile kt - 1 occupied, whose last reads completed before the preceding
// barrier, and is first read in the phase after the last of them.  Sums run in
// the same order as in k_dqgemm, so the two give identical bits.
__device__ __forceinline__ void phase_end() {
  __builtin_amdgcn_sched_barrier(0);
  __syncthreads();
  __builtin_amdgcn_sched_barrier(0);
}

// SPLIT: workgroup w takes K-steps [s KT / splits, (s + 1) KT / splits) of
// tile w mod T (s = w / T) and adds its partial tile into y, which the host
// has zeroed; used when the tiles alone would leave much of the GPU idle in
// the last round.
// TI = 2: 128 x 256 tiles (each wave 64 x 64) for 65-128 rows, where a
// 256-row tile would multiply zero rows half the time.
template <int XT, bool SPLIT, int TI = 4>
__global__ void __launch_bounds__(512) k_dqgemm_pp(const uint16_t* __restrict__ x, const int8_t* __restrict__ codes,
                                                  const float* __restrict__ scales, int64_t M, int64_t N, int64_t K,
                                                  int lgB, float* __restrict__ y, int64_t mtiles, int64_t ntiles,
                                                  int splits) {
  constexpr int BM = 64 * TI, BN = 256, WN = 4, NT = 512;
  constexpr int TJ = 2;                          // 32 x 32 MFMA tiles per wave: TI x 2 (128 or 64 x 64)
  constexpr int XC = BM * kBK / 8 / NT;          // x chunks per thread and K-step (TI)
  constexpr int WC = BN * kBK / 16 / NT;         // 2 code chunks per thread and K-step
  constexpr int XH = XC / 2;                     // x chunks per part
  static_assert((TI == 4 || TI == 2) && XC == TI && WC == 2, "tile shape");
  __shared__ u32x4 As[2][BM * kLDK / 8];
  __shared__ u32x4 Bs[2][BN * kLDK / 8];

  const int64_t T = mtiles * ntiles;
  const int64_t wg = SPLIT ? blockIdx.x % T : blockIdx.x;
  const int64_t q = T / kXcds, r = T % kXcds, xcd = wg % kXcds, idx = wg / kXcds;
  const int64_t t = !ZQ_GEMM_XCD_MAP ? wg : xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
  const int64_t per_group = (int64_t)kGroupM * ntiles;
  const int64_t first_m = (t / per_group) * kGroupM;
  const int64_t gsize = mtiles - first_m < kGroupM ? mtiles - first_m : kGroupM;
  const int64_t mt = first_m + (t % per_group) % gsize;
  const int64_t nt = (t % per_group) / gsize;
  const int64_t m0 = mt * BM, n0 = nt * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, wm = wave / WN, wn = wave % WN;
  const int KTall = (int)(K / kBK);
  const int split = SPLIT ? (int)(blockIdx.x / T) : 0;
  const int kt0 = SPLIT ? (int)((int64_t)split * KTall / splits) : 0;
  const int KT = SPLIT ? (int)((int64_t)(split + 1) * KTall / splits) - kt0 : KTall;

  // tile kt + 1 is held in registers from its loads (phases of K-step kt - 1)
  // to its LDS store (phases of K-step kt): part P of a tile is x chunks 2P,
  // 2P + 1 and code chunk P of each thread, stored and then reloaded with the
  // next tile's part in the same phase, which leaves each load a whole K-step
  // (four phases) to arrive
  u32x4 xrs[1][XC], wrs[1][WC];
  float srs[1][WC];
  // Loads are buffer loads: a wave-uniform resource per operand (base at the
  // tile's first row, size up to the operand's last row in the tile) plus
  // loop-invariant 32-bit lane offsets (the host keeps K <= kDqGemmPpMaxK, so
  // 256 rows of 2 K bytes fit) and the K-step's byte offset in a scalar
  // register.  Rows past M (columns past N) of a ragged edge tile fall
  // outside the resource and read as zero; they only enter outputs that are
  // never stored.  The scales' base index n0 K / B is exact because n0 K is a
  // multiple of 256 * 64 >= B.
  uint32_t xoff[XC], woff[WC];
#pragma unroll
  for (int i = 0; i < XC; ++i) {
    const int c = tid + NT * i, row = c >> 3, col = (c & 7) * 8;
    xoff[i] = (uint32_t)((row * K + col) * 2);
  }
#pragma unroll
  for (int i = 0; i < WC; ++i) {
    const int c = tid + NT * i, row = c >> 2, col = (c & 3) * 16;
    woff[i] = (uint32_t)(row * K + col);
  }
  const int64_t mrows = M - m0 < BM ? M - m0 : BM, nrows = N - n0 < BN ? N - n0 : BN;
  const __amdgpu_buffer_rsrc_t xres =
      __builtin_amdgcn_make_buffer_rsrc((void*)(x + m0 * K), (short)0, (int)(mrows * K * 2), kBufferFlags);
  const __amdgpu_buffer_rsrc_t wres =
      __builtin_amdgcn_make_buffer_rsrc((void*)(codes + n0 * K), (short)0, (int)(nrows * K), kBufferFlags);
  const int64_t s0 = (n0 * K) >> lgB, s1 = ((n0 + nrows) * K + (1 << lgB) - 1) >> lgB;
  const __amdgpu_buffer_rsrc_t sres =
      __builtin_amdgcn_make_buffer_rsrc((void*)(scales + s0), (short)0, (int)((s1 - s0) * 4), kBufferFlags);
  auto gload = [&](int kt, auto part_c) {
    constexpr int R = 0, P = decltype(part_c)::value;
    const int k0 = (kt0 + kt) * kBK;
#pragma unroll
    for (int i = XH * P; i < XH * P + XH; ++i)
      xrs[R][i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(xres, (int)xoff[i], 2 * k0, 0));
    wrs[R][P] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(wres, (int)woff[P], k0, 0));
    const uint32_t si = (woff[P] + (uint32_t)k0) >> lgB;
    srs[R][P] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(sres, (int)(si * 4), 0, 0));
  };
  // part P of the register tile: its 16 codes become fl(q * s) narrowed to
  // XT in ob (deq), then x's chunks and ob go to LDS buffer `buf` (store)
  uint32_t ob[8];
  auto deq = [&](auto part_c) {
    constexpr int P = decltype(part_c)::value;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t word = wrs[0][P][j >> 1];
      const int sh = (j & 1) * 16;
      const float v0 = (float)(int32_t)(int8_t)(word >> sh) * srs[0][P];
      const float v1 = (float)(int32_t)(int8_t)(word >> (sh + 8)) * srs[0][P];
      ob[j] = narrow2<XT>(v0, v1);
    }
  };
  auto store = [&](int buf, auto part_c) {
    constexpr int P = decltype(part_c)::value;
#pragma unroll
    for (int i = XH * P; i < XH * P + XH; ++i) {
      const int c = tid + NT * i;
      As[buf][(c >> 3) * kRow16 + (c & 7)] = xrs[0][i];
    }
    const int c = tid + NT * P, bi = (c >> 2) * kRow16 + (c & 3) * 2;
    Bs[buf][bi] = u32x4{ob[0], ob[1], ob[2], ob[3]};
    Bs[buf][bi + 1] = u32x4{ob[4], ob[5], ob[6], ob[7]};
  };

  f32x16_t acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  // operand fragments of one half K-step: k steps 2H and 2H + 1 of 16
  // (LDS indices in 16-byte units: a row is kRow16 of them, so the
  // per-fragment offsets are constants)
  const int frow = lane & 31;
  const int abase = (wm * TI * 32 + frow) * kRow16 + (lane >> 5), bbase = (wn * TJ * 32 + frow) * kRow16 + (lane >> 5);
  u32x4 fa[TI][2], fb[TJ][2];
  auto read_frags = [&](int buf, auto half_c) {
    constexpr int H = decltype(half_c)::value;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int kk = 2 * H + s;
#pragma unroll
      for (int i = 0; i < TI; ++i) fa[i][s] = As[buf][abase + i * 32 * kRow16 + kk * 2];
#pragma unroll
      for (int j = 0; j < TJ; ++j) fb[j][s] = Bs[buf][bbase + j * 32 * kRow16 + kk * 2];
    }
  };
  // the 16 MFMAs of a half K-step; with DQ, the dequantisation of code part
  // P is interleaved with them (the matrix core runs each MFMA for 32 cycles,
  // in which this wave's own VALU is otherwise idle).  Both wave groups keep
  // the default priority: raising it for the MFMA phase measured 3-8% slower.
  auto mma = [&](auto part_c, auto dq_c) {
    constexpr int P = decltype(part_c)::value;
    constexpr bool DQ = decltype(dq_c)::value;
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) acc[i][j] = mfma32<XT>(fa[i][s], fb[j][s], acc[i][j]);
    if constexpr (DQ && TI == 4) {
      deq(part_c);
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);  // 4 MFMAs first: the codes may still be arriving
#pragma unroll
      for (int q = 0; q < 10; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // 1 MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);  // 4 VALU
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    } else if constexpr (DQ) {
      deq(part_c);  // 8 MFMAs: the same 40 VALU instructions, 8 after each of 5
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
#pragma unroll
      for (int q = 0; q < 5; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
    (void)P;
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  // K-step kt from LDS buffer kt % 2.  With ST, tile kt + 1 goes from the
  // registers into the other buffer (part 0 in the first memory phase, part 1
  // in the second; each B part was dequantised during the preceding MFMA
  // phase), and with LD tile kt + 2 is loaded into the registers (part P at
  // the start of the MFMA phase after part P of tile kt + 1 left them) and its
  // part 0 dequantised.  The steady-state loop has both and no branches, so
  // each wait covers exactly the loads it needs.
  auto kstep = [&](int kt, auto st_c, auto ld_c) {
    constexpr bool ST = decltype(st_c)::value, LD = decltype(ld_c)::value;
    const int cur = kt & 1;
    if constexpr (ST) store(cur ^ 1, I0{});
    read_frags(cur, I0{});
    phase_end();
    if constexpr (LD) gload(kt + 2, I0{});
    mma(I1{}, st_c);
    phase_end();
    if constexpr (ST) store(cur ^ 1, I1{});
    read_frags(cur, I1{});
    phase_end();
    if constexpr (LD) gload(kt + 2, I1{});
    mma(I0{}, ld_c);
    phase_end();
  };
  using T_ = std::true_type;
  using F_ = std::false_type;

  if (KT > 0) {
    gload(0, I0{});
    gload(0, I1{});
    deq(I0{});
    store(0, I0{});
    deq(I1{});
    store(0, I1{});
  }
  // the loads of tile 1 in the loop's order (part 0, then part 1), so that
  // the wait counts at the loop head are those of the steady state; its
  // part 0 is dequantised here, as the loop does for the tiles after it
  if (KT > 1) {
    __builtin_amdgcn_sched_barrier(0);
    gload(1, I0{});
    __builtin_amdgcn_sched_barrier(0);
    gload(1, I1{});
    __builtin_amdgcn_sched_barrier(0);
    deq(I0{});
  }
  __syncthreads();
  if (wm == 1) phase_end();  // the second wave group starts one phase later
  int kt = 0;
#pragma unroll 1
  for (; kt + 2 < KT; ++kt) kstep(kt, T_{}, T_{});
  if (kt + 1 < KT) kstep(kt++, T_{}, F_{});
  if (kt < KT) kstep(kt, F_{}, F_{});
  if (wm == 0) phase_end();  // ... and the first one waits for its last phase

#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int64_t n = n0 + wn * TJ * 32 + j * 32 + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t m = m0 + wm * TI * 32 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (m < M && n < N) {
          if constexpr (SPLIT) atomicAdd(y + m * N + n, acc[i][j][e]);
          else y[m * N + n] = acc[i][j][e];
        }
      }
    }
}

// Few tokens (M <= kGemvRows): a weight-streaming kernel on
// v_mfma_f32_16x16x32.  Workgroup (g, s) takes weight rows [64 g, 64 g + 64),
// 16 per wave, and the K range [s kc, min(K, (s + 1) kc)), kc <= kGemvKc.
// Within each 256-wide chunk of that range, lane l (row l % 16 of its wave's
// 16, lane group h = l / 16) loads the 64 codes k = 64 h .. 64 h + 63 of its
// row straight from memory, and its 8 operand codes of MFMA t are
// k = 64 h + 8 t .. 64 h + 8 t + 7; x's fragments are read from LDS with the
// same mapping, so each MFMA sums the same products as the plain order would,
// grouped differently.  All chunks of a wave's range are loaded before any is
// used (16 KB per wave), x's rows over the range are staged into LDS once,
// and the loop has no barrier.  Rows M .. 15 of the x slab, and its columns
// past the range, are zero.
constexpr int kGemvRows = 16;   // x rows (M <= kGemvRows)
constexpr int kGemvKc = 1024;   // longest K range of a workgroup

template <int XT>
__device__ __forceinline__ f32x4_t mfma16(u32x4 a, u32x4 b, f32x4_t c) {
  if constexpr (XT == ZQ_BF16)
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b), c,
                                                  0, 0, 0);
}

template <int XT, bool SPLIT>
__global__ void __launch_bounds__(256) k_dqgemv(const uint16_t* __restrict__ x, const int8_t* __restrict__ codes,
                                                const float* __restrict__ scales, int64_t M, int64_t N, int64_t K,
                                                int lgB, float* __restrict__ y, int64_t ngroups, int kc) {
  constexpr int NC = kGemvKc / 256, G16 = kGemvKc / 8;  // chunks per wave at most; 16-byte granules per slab row
  // x slab: row m, granule q (elements 8 q .. 8 q + 7 of the range) at
  // m * G16 + (q ^ m): the 16 rows' granules of one fragment read then fall
  // in 16 distinct 16-byte bank groups
  __shared__ u32x4 xs[kGemvRows * G16];
  const int64_t grp = blockIdx.x % ngroups, split = blockIdx.x / ngroups;
  const int64_t kb = split * kc, ke = K - kb < kc ? K : kb + kc;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, r = lane & 15, h = lane >> 4;
  const int64_t n = grp * 64 + wave * 16 + r;

  // codes and scales of every chunk (a 64-code segment is 64-aligned in the
  // flat index, so it spans at most two blocks of B >= 32: codes 0-31 and
  // 32-63 take scales 0 and 1)
  u32x4 cw[NC][4];
  float sc[NC][2];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int64_t k = kb + 256 * c + 64 * h;
    if (n < N && k < ke) {
      const int64_t f = n * K + k;
      const u32x4* p = reinterpret_cast<const u32x4*>(codes + f);
#pragma unroll
      for (int j = 0; j < 4; ++j) cw[c][j] = p[j];
      sc[c][0] = scales[f >> lgB];
      sc[c][1] = scales[(f + 32) >> lgB];
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) cw[c][j] = u32x4{0u, 0u, 0u, 0u};
      sc[c][0] = sc[c][1] = 0.0f;
    }
  }
  // every granule of the slab is written (zero past the range), so the
  // fragments of a partly covered chunk read zeros, never stale LDS
  for (int i = tid; i < kGemvRows * G16; i += 256) {
    const int m = i / G16, q = i % G16;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (m < M && kb + 8 * q < ke) v = *reinterpret_cast<const u32x4*>(x + m * K + kb + 8 * q);
    xs[m * G16 + (q ^ m)] = v;
  }
  __syncthreads();

  f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    if (kb + 256 * c >= ke) break;  // workgroup-uniform
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const u32x4 wv = cw[c][t >> 1];
      const uint32_t w0 = (t & 1) ? wv.z : wv.x, w1 = (t & 1) ? wv.w : wv.y;
      const float s = sc[c][t >> 2];
      uint32_t b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t w = u < 2 ? w0 : w1;
        const int sh = (u & 1) * 16;
        const float v0 = (float)(int32_t)(int8_t)(w >> sh) * s;
        const float v1 = (float)(int32_t)(int8_t)(w >> (sh + 8)) * s;
        b[u] = narrow2<XT>(v0, v1);
      }
      const int q = 32 * c + 8 * h + t;
      acc = mfma16<XT>(xs[r * G16 + (q ^ r)], u32x4{b[0], b[1], b[2], b[3]}, acc);
    }
  }
  // D register e of lane l: row 4 (l / 16) + e, column l % 16
  if (n < N) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t m = 4 * h + e;
      if (m < M) {
        if constexpr (SPLIT) atomicAdd(y + m * N + n, acc[e]);
        else y[m * N + n] = acc[e];
      }
    }
  }
}

// y[0, count) = 0 (for the split kernel, which adds into y)
__global__ void __launch_bounds__(256) k_fill_zero(float* __restrict__ y, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (int64_t)gridDim.x * 256) y[i] = 0.0f;
}

static_assert(!ZQ_GEMM_PINGPONG || (kDqGemmTileM == 256 && kDqGemmTileN == 256 && kDqGemmThreads == 512), "ping-pong tile");
static_assert(64 * ZQ_GEMM_WM * ZQ_GEMM_WN == kDqGemmThreads, "launch shape");

// pp: the ping-pong kernel (K <= kDqGemmPpMaxK), with 128-row tiles if half;
// otherwise the plain 256 x 256 kernel, which never splits K
DqGemmKernel dqgemm_kernel(int xt, bool split, bool pp, bool half) {
  if (pp && half) {
    if (split) return xt == ZQ_BF16 ? &k_dqgemm_pp<ZQ_BF16, true, 2> : &k_dqgemm_pp<ZQ_F16, true, 2>;
    return xt == ZQ_BF16 ? &k_dqgemm_pp<ZQ_BF16, false, 2> : &k_dqgemm_pp<ZQ_F16, false, 2>;
  }
  if (pp) {
    if (split) return xt == ZQ_BF16 ? &k_dqgemm_pp<ZQ_BF16, true> : &k_dqgemm_pp<ZQ_F16, true>;
    return xt == ZQ_BF16 ? &k_dqgemm_pp<ZQ_BF16, false> : &k_dqgemm_pp<ZQ_F16, false>;
  }
  return xt == ZQ_BF16 ? &k_dqgemm<ZQ_BF16, kDqGemmTileM, kDqGemmTileN, ZQ_GEMM_WM, ZQ_GEMM_WN>
                       : &k_dqgemm<ZQ_F16, kDqGemmTileM, kDqGemmTileN, ZQ_GEMM_WM, ZQ_GEMM_WN>;
}

// K splits for the 256 x 256 tiles.  A tile's workgroup fills a CU (its LDS
// buffers alone take 147 KB), so the tiles run in rounds of one workgroup per
// CU, and a last round that is mostly empty idles much of the GPU (72 tiles
// on 256 CUs use 28% of it).  Splitting K s ways makes s times as many
// workgroups of 1/s the K-steps, at the price of a zero fill of y and
// M N s atomic additions; the count taken minimises the modelled time
//   ceil(tiles s / CUs) ceil(ksteps / s) step  +  [s > 1] M N s atomic
// (step, atomic: ZQ_GEMM_PP_STEP_NS, ZQ_GEMM_ATOMIC_PS), which splits the
// GEMMs of a few hundred rows 2-16 ways and leaves full rounds whole.
int64_t large_splits(int64_t tiles, int64_t ksteps, int64_t M, int64_t N, double step_scale) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  const int64_t most = ksteps < kDqGemmMaxSplits ? ksteps : kDqGemmMaxSplits;
  const double step = ZQ_GEMM_PP_STEP_NS * 1e-9 * step_scale, atomic = ZQ_GEMM_ATOMIC_PS * 1e-12;
  auto cost = [&](int64_t s) {
    const double rounds = (double)((tiles * s + cus - 1) / cus), steps = (double)((ksteps + s - 1) / s);
    return rounds * steps * step + (s > 1 ? (double)M * (double)N * (double)s * atomic : 0.0);
  };
  int64_t best = 1;
  double best_cost = cost(1);
  for (int64_t s = 2; s <= most; ++s) {
    const double c = cost(s);
    if (c < best_cost) {
      best = s;
      best_cost = c;
    }
  }
  return best;
}

}  // namespace
}  // namespace zq

using namespace zq;

// qwz_dequant_gemm (include/zq.h): argument checks, then one launch (or a
// zero fill and a split-K launch when the tiles are few)
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
  if (M <= kGemvRows) {
    // few tokens: the weight-streaming kernel; the K range per workgroup
    // halves (down to 256) until about kGemvTargetWgs workgroups run
    const int64_t ngroups = (N + 63) / 64;
    int64_t kc = kGemvKc;
    while (kc > 256 && ngroups * ((K + kc - 1) / kc) < kGemvTargetWgs) kc /= 2;
    const int64_t splits = K > kc ? (K + kc - 1) / kc : 1;
    if (ngroups * splits > kMaxGrid) return ZQ_E_SIZE;
    if (splits == 1)
      return launch(xt == ZQ_BF16 ? &k_dqgemv<ZQ_BF16, false> : &k_dqgemv<ZQ_F16, false>, (unsigned)ngroups, 256u, st,
                    xh, codes, scales, M, N, K, lgB, y, ngroups, (int)kc);
    const int64_t count = M * N, fill_grid = count / 256 + 1 < 4096 ? count / 256 + 1 : 4096;
    int rc = launch(&k_fill_zero, (unsigned)fill_grid, 256u, st, y, count);
    if (rc != ZQ_OK) return rc;
    return launch(xt == ZQ_BF16 ? &k_dqgemv<ZQ_BF16, true> : &k_dqgemv<ZQ_F16, true>, (unsigned)(ngroups * splits),
                  256u, st, xh, codes, scales, M, N, K, lgB, y, ngroups, (int)kc);
  }
  // the ping-pong kernel, K split where its tiles are few; up to
  // ZQ_GEMM_HALF_M rows with 128 x 256 tiles (a K-step of one costs about 0.6
  // of a 256 x 256 tile's: half the MFMAs, the same dequantisation)
  const bool pp = ZQ_GEMM_PINGPONG && K <= kDqGemmPpMaxK, half = pp && M <= ZQ_GEMM_HALF_M;
  const int64_t bm = half ? kDqGemmTileM / 2 : kDqGemmTileM;
  const int64_t mtiles = (M + bm - 1) / bm, ntiles = (N + kDqGemmTileN - 1) / kDqGemmTileN;
  const int64_t tiles = mtiles * ntiles;
  const int64_t splits = pp ? large_splits(tiles, K / kDqGemmK, M, N, half ? 0.6 : 1.0) : 1;
  if (tiles * splits > kMaxGrid) return ZQ_E_SIZE;
  if (splits > 1) {
    const int64_t count = M * N, fill_grid = count / 256 + 1 < 4096 ? count / 256 + 1 : 4096;
    int rc = launch(&k_fill_zero, (unsigned)fill_grid, 256u, st, y, count);
    if (rc != ZQ_OK) return rc;
  }
  return launch(dqgemm_kernel(xt, splits > 1, pp, half), (unsigned)(tiles * splits), kDqGemmThreads, st, xh, codes,
                scales, M, N, K, lgB, y, mtiles, ntiles, (int)splits);
}
