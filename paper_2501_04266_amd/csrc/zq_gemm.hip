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
// Tiling: a workgroup of 8 waves computes a 256 x 256 tile of y, each wave a
// 128 x 64 block as 4 x 2 MFMA tiles of 32 x 32 (other shapes are template
// parameters).  K advances 64 at a time.  x tiles (16 B per load) and code
// tiles (16 codes and their scale per load) are fetched into one of two
// register sets two K-steps ahead, so a load has a whole K-step of MFMAs to
// arrive in; at the end of each K-step the next tile is dequantised and
// stored into the LDS buffer not being read.  LDS rows are padded by 16 bytes so the 16-byte
// fragment reads of 8 consecutive lanes fall in distinct banks.  Workgroups
// are numbered so that each XCD receives a contiguous range of tiles, and
// within it groups of 4 tile rows share their weight tiles through that XCD's
// L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "zq.h"
#include "zq_device.h"
#include "zq_internal.h"

#pragma clang fp contract(off)

namespace zq {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kBK = 64;
constexpr int kLDK = kBK + 8;  // LDS row stride in 16-bit elements (144 bytes)
#ifndef ZQ_GEMM_GROUP_M
#define ZQ_GEMM_GROUP_M 4
#endif
#ifndef ZQ_GEMM_XCD_MAP
#define ZQ_GEMM_XCD_MAP 1
#endif
constexpr int kGroupM = ZQ_GEMM_GROUP_M;  // tile rows sharing a weight tile in L2
constexpr int kXcds = 8;

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
// block of 32 x 32 MFMA tiles.
// SPLIT: workgroup w takes K-steps [s KT / splits, (s + 1) KT / splits) of
// tile w / splits (s = w % splits) and adds its partial tile into y, which the
// host has zeroed; used when there are too few tiles to fill the GPU.
template <int XT, int BM, int BN, int WM, int WN, bool SPLIT>
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
  const int64_t wg = SPLIT ? blockIdx.x / splits : blockIdx.x;
  const int64_t q = T / kXcds, r = T % kXcds, xcd = wg % kXcds, idx = wg / kXcds;
  const int64_t t = SPLIT || !ZQ_GEMM_XCD_MAP ? wg : xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
  const int64_t per_group = (int64_t)kGroupM * ntiles;
  const int64_t first_m = (t / per_group) * kGroupM;
  const int64_t gsize = mtiles - first_m < kGroupM ? mtiles - first_m : kGroupM;
  const int64_t mt = first_m + (t % per_group) % gsize;
  const int64_t nt = (t % per_group) / gsize;
  const int64_t m0 = mt * BM, n0 = nt * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, wm = wave / WN, wn = wave % WN;
  const int KTall = (int)(K / kBK);
  const int split = SPLIT ? (int)(blockIdx.x % splits) : 0;
  const int kt0 = SPLIT ? (int)((int64_t)split * KTall / splits) : 0;
  const int KT = SPLIT ? (int)((int64_t)(split + 1) * KTall / splits) - kt0 : KTall;

  // RS register sets: with 2, tile t's loads are issued two K-steps before
  // its LDS store
  constexpr int RS = ZQ_GEMM_RSETS;
  u32x4 xrs[RS][XC], wrs[RS][WC];
  float srs[RS][WC];
  // global -> registers: x rows m0.., 8 elements per chunk; codes rows n0..,
  // 16 codes per chunk with the scale of their block (a chunk never straddles
  // a block: chunks are 16-aligned in the flat index and B >= 32)
  auto gload = [&](int kt, auto rs_c) {
    constexpr int R = decltype(rs_c)::value;
    u32x4(&xr)[XC] = xrs[R];
    u32x4(&wr)[WC] = wrs[R];
    float(&sr)[WC] = srs[R];
    const int64_t k0 = (int64_t)(kt0 + kt) * kBK;
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
  using R1 = std::integral_constant<int, RS - 1>;
  if constexpr (RS == 1) {
    if (KT > 0) {
      gload(0, R0{});
      sstore(0, R0{});
    }
    __syncthreads();
#pragma unroll 1
    for (int kt = 0; kt < KT; ++kt) {
      const int cur = kt & 1;
      if (kt + 1 < KT) gload(kt + 1, R0{});
      compute(cur);
      if (kt + 1 < KT) sstore(cur ^ 1, R0{});
      __syncthreads();
    }
  } else {
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
        if (m < M && n < N) {
          if constexpr (SPLIT) atomicAdd(y + m * N + n, acc[i][j][e]);
          else y[m * N + n] = acc[i][j][e];
        }
      }
    }
}

// y[0, count) = 0 (for the split kernel, which adds into y)
__global__ void __launch_bounds__(256) k_fill_zero(float* __restrict__ y, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (int64_t)gridDim.x * 256) y[i] = 0.0f;
}

}  // namespace

static_assert(64 * ZQ_GEMM_WM * ZQ_GEMM_WN == kDqGemmThreads && 64 * 2 * 2 == kDqGemmSmallThreads, "launch shape");

DqGemmKernel dqgemm_kernel(int xt, bool small, bool split) {
  if (!small)
    return xt == ZQ_BF16 ? &k_dqgemm<ZQ_BF16, kDqGemmTileM, kDqGemmTileN, ZQ_GEMM_WM, ZQ_GEMM_WN, false>
                         : &k_dqgemm<ZQ_F16, kDqGemmTileM, kDqGemmTileN, ZQ_GEMM_WM, ZQ_GEMM_WN, false>;
  if (split)
    return xt == ZQ_BF16 ? &k_dqgemm<ZQ_BF16, kDqGemmSmallTile, kDqGemmSmallTile, 2, 2, true>
                         : &k_dqgemm<ZQ_F16, kDqGemmSmallTile, kDqGemmSmallTile, 2, 2, true>;
  return xt == ZQ_BF16 ? &k_dqgemm<ZQ_BF16, kDqGemmSmallTile, kDqGemmSmallTile, 2, 2, false>
                       : &k_dqgemm<ZQ_F16, kDqGemmSmallTile, kDqGemmSmallTile, 2, 2, false>;
}

FillZeroKernel fill_zero_kernel() { return &k_fill_zero; }

}  // namespace zq
