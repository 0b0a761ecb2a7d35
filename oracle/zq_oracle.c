/*
 * zq_oracle.c -- plain CPU oracle of the qwZ / qgZ compression data path.
 *
 * TEST INFRASTRUCTURE ONLY.  The test-suite, the smoke check and the
 * benchmark's CPU-baseline leg are the only callers.  The product library
 * (HIP kernels behind include/zq.h) shares no code, header, table or helper
 * with this file and never calls it.
 *
 * Method (arXiv 2501.04266, "Scaling Large Language Model Training on
 * Frontier with Low-Bandwidth Partitioning"):
 *   - Background, ZeRO++ subsection: ZeRO++ quantises fp16 data block-wise
 *     into INT8 blocks for the weight Allgather (qwZ, halves its volume) and
 *     into INT4 blocks for the gradient all-to-all reduce-scatter (qgZ,
 *     quarters its volume).  In that reduce-scatter the receiver of P slices
 *     dequantises them, sums them and quantises the sum again.
 *   - Design, Weight Partitioning: the ZeRO++ quantiser and dequantiser run
 *     around each Allgather; the secondary weight partition is stored in the
 *     quantised format.
 *   - Design, Communication Volume Analysis: one INT8 byte replaces two FP16
 *     bytes per weight; INT4 cuts the gradient volume four-fold.
 *   - Evaluations, Model Convergence: every block carries its own scale
 *     (block-wise quantisation after Dettmers et al.).
 *
 * The paper states no formula.  The readings used here, each marked at the
 * step it governs, are: symmetric absmax scaling with code range +-qmax
 * (qmax = 127 for INT8, 7 for INT4); the stored scale is a/qmax and codes are
 * made by multiplying with the correctly rounded reciprocal qmax/a; rounding
 * is to nearest with ties to even; a block whose absmax is below 2^-119
 * (including an all-zero block) gets scale 0 and all-zero codes; the last
 * block of a tensor may be short and uses only its own elements; INT4 codes
 * are two's-complement nibbles, even element in the low nibble; scales are
 * binary32; the P-slice sum starts at +0 and adds the slices in ascending
 * order, one rounded multiply then one rounded add per slice (no fused
 * multiply-add).
 *
 * Arithmetic: built with -O2 -fno-fast-math -ffp-contract=off for x86-64,
 * where float expressions are evaluated in binary32 (SSE), so each float
 * operation below is exactly one correctly rounded IEEE binary32 operation.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ZQO_F32 = 0, ZQO_F16 = 1, ZQO_BF16 = 2 };
enum {
  ZQO_OK = 0,
  ZQO_E_ARG = -1,      /* null pointer, bad dtype, block or P */
  ZQO_E_RANGE = -2     /* a code fell outside +-qmax (impossible for finite input) */
};

#define ZQO_MAX_BLOCK 4096

/* ------------------------------------------------------------------ */
/* Element formats                                                     */
/* ------------------------------------------------------------------ */

static float f32_of_bits(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t bits_of_f32(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

/* binary16 -> binary32, exact, straight from the binary16 encoding:
 * subnormal  m * 2^-24,  normal (1024 + m) * 2^(e - 25). */
static float f16_to_f32(uint16_t h) {
  int sign = h >> 15, e = (h >> 10) & 31, m = h & 1023;
  float v;
  if (e == 0) v = ldexpf((float)m, -24);
  else if (e == 31) v = m ? NAN : INFINITY;
  else v = ldexpf((float)(m + 1024), e - 25);
  return sign ? -v : v;
}

/* bfloat16 is the upper half of a binary32: widening is exact. */
static float bf16_to_f32(uint16_t h) { return f32_of_bits((uint32_t)h << 16); }

/* binary32 -> bfloat16, round to nearest, ties to even, on the 16 dropped
 * bits.  A carry out of the kept mantissa moves into the exponent, which is
 * the correct next value (up to infinity). */
static uint16_t f32_to_bf16(float f) {
  uint32_t u = bits_of_f32(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  uint32_t upper = u >> 16, dropped = u & 0xffffu;
  if (dropped > 0x8000u || (dropped == 0x8000u && (upper & 1u))) upper += 1u;
  return (uint16_t)upper;
}

/* binary32 -> binary16, round to nearest, ties to even.  The binary16 grid
 * near |f| has spacing 2^(E-10) for |f| in [2^E, 2^(E+1)), E >= -14, and
 * 2^-24 below 2^-14 (subnormals).  |f| / spacing is exact in binary64;
 * nearbyint rounds it half-to-even. |f| >= 65520 (max + half a step) is
 * infinity. */
static uint16_t f32_to_f16(float f) {
  uint16_t sign = (uint16_t)((bits_of_f32(f) >> 16) & 0x8000u);
  float a = fabsf(f);
  if (isnan(f)) return (uint16_t)(sign | 0x7e00u);
  if (a >= 65520.0f) return (uint16_t)(sign | 0x7c00u);
  if (a == 0.0f) return sign;
  int e2;
  frexpf(a, &e2);                       /* a in [2^(e2-1), 2^e2) */
  int E = e2 - 1;
  if (E < -14) E = -14;
  double spacing = ldexp(1.0, E - 10);
  double k = nearbyint((double)a / spacing);
  double v = k * spacing;
  if (v < ldexp(1.0, -14)) return (uint16_t)(sign | (uint16_t)k);  /* subnormal */
  int ve;
  frexp(v, &ve);                        /* rounding may reach the next binade */
  int Ev = ve - 1;
  uint16_t mant = (uint16_t)(ldexp(v, 10 - Ev) - 1024.0);
  return (uint16_t)(sign | (uint16_t)((Ev + 15) << 10) | mant);
}

static float load_elem(const void* x, int dt, int64_t i) {
  switch (dt) {
    case ZQO_F32: return ((const float*)x)[i];
    case ZQO_F16: return f16_to_f32(((const uint16_t*)x)[i]);
    default: return bf16_to_f32(((const uint16_t*)x)[i]);
  }
}

static void store_elem(void* y, int dt, int64_t i, float v) {
  switch (dt) {
    case ZQO_F32: ((float*)y)[i] = v; break;
    case ZQO_F16: ((uint16_t*)y)[i] = f32_to_f16(v); break;
    default: ((uint16_t*)y)[i] = f32_to_bf16(v); break;
  }
}

/* two's-complement INT4 nibble k of a packed stream: element 2j is the low
 * nibble of byte j, element 2j+1 the high nibble. */
static int nibble_at(const uint8_t* packed, int64_t k) {
  int v = (k & 1) ? (packed[k >> 1] >> 4) : (packed[k >> 1] & 0x0f);
  return v >= 8 ? v - 16 : v;
}

/* ------------------------------------------------------------------ */
/* One block: absmax, scale, codes                                     */
/* ------------------------------------------------------------------ */

/* Symmetric block quantisation of len binary32 values (ZeRO++ block-based
 * quantisation, Background; per-block scale, Model Convergence).
 *   a = max |v_i|                      (exact, so order is irrelevant)
 *   a < 2^-119  ->  scale 0, codes 0   (zero-block reading; keeps qmax/a
 *                                       finite and the scale normal)
 *   scale = fl(a / qmax),  r = fl(qmax / a)
 *   code_i = nearest integer to fl(v_i * r), ties to even.
 * |fl(v_i * r)| <= qmax (1 + 2^-24)^2 < qmax + 1/2, so no code leaves
 * [-qmax, qmax]; the check below only guards that argument. */
static int quantize_block(const float* v, int64_t len, int qmax, int* q, float* scale) {
  float a = 0.0f;
  for (int64_t i = 0; i < len; ++i) {
    float m = fabsf(v[i]);
    if (m > a) a = m;
  }
  if (a < 0x1p-119f) {
    for (int64_t i = 0; i < len; ++i) q[i] = 0;
    *scale = 0.0f;
    return ZQO_OK;
  }
  float s = a / (float)qmax;
  float r = (float)qmax / a;
  for (int64_t i = 0; i < len; ++i) {
    float t = v[i] * r;
    float k = nearbyintf(t);
    if (k > (float)qmax || k < -(float)qmax) return ZQO_E_RANGE;
    q[i] = (int)k;
  }
  *scale = s;
  return ZQO_OK;
}

static int block_ok(int32_t block) { return block >= 2 && block <= ZQO_MAX_BLOCK && (block % 2) == 0; }
static int dtype_ok(int dt) { return dt == ZQO_F32 || dt == ZQO_F16 || dt == ZQO_BF16; }
static int64_t nblocks(int64_t n, int32_t block) { return (n + block - 1) / block; }

/* ------------------------------------------------------------------ */
/* Public oracle calls                                                 */
/* ------------------------------------------------------------------ */

void zqo_set_threads(int t) {
#ifdef _OPENMP
  if (t > 0) omp_set_num_threads(t);
#else
  (void)t;
#endif
}

int zqo_get_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* qwZ quantiser: x[n] (f32 / f16 / bf16) -> INT8 codes[n] + scales[ceil(n/B)]. */
int zqo_qwz_quantize(const void* x, int xt, int64_t n, int32_t block, int8_t* codes, float* scales) {
  if (n < 0 || !block_ok(block) || !dtype_ok(xt)) return ZQO_E_ARG;
  if (n == 0) return ZQO_OK;
  if (!x || !codes || !scales) return ZQO_E_ARG;
  int64_t nb = nblocks(n, block);
  int status = ZQO_OK;
#pragma omp parallel for schedule(static) reduction(min : status)
  for (int64_t b = 0; b < nb; ++b) {
    float v[ZQO_MAX_BLOCK];
    int q[ZQO_MAX_BLOCK];
    int64_t base = b * block, len = n - base < block ? n - base : block;
    for (int64_t i = 0; i < len; ++i) v[i] = load_elem(x, xt, base + i);
    if (quantize_block(v, len, 127, q, &scales[b]) != ZQO_OK) status = ZQO_E_RANGE;
    for (int64_t i = 0; i < len; ++i) codes[base + i] = (int8_t)q[i];
  }
  return status;
}

/* qwZ dequantiser: y_i = cvt(fl(code_i * scale_b)), cvt = identity or
 * round-to-nearest-even narrowing to f16 / bf16. */
int zqo_qwz_dequantize(const int8_t* codes, const float* scales, int64_t n, int32_t block, void* y, int yt) {
  if (n < 0 || !block_ok(block) || !dtype_ok(yt)) return ZQO_E_ARG;
  if (n == 0) return ZQO_OK;
  if (!codes || !scales || !y) return ZQO_E_ARG;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    float prod = (float)codes[i] * scales[i / block];
    store_elem(y, yt, i, prod);
  }
  return ZQO_OK;
}

/* qgZ quantiser: g[n] -> packed INT4 bytes[ceil(n/2)] + scales[ceil(n/B)].
 * B is even, so every block starts on a byte boundary.  For odd n the high
 * nibble of the last byte is 0. */
int zqo_qgz_quantize(const void* g, int gt, int64_t n, int32_t block, uint8_t* packed, float* scales) {
  if (n < 0 || !block_ok(block) || !dtype_ok(gt)) return ZQO_E_ARG;
  if (n == 0) return ZQO_OK;
  if (!g || !packed || !scales) return ZQO_E_ARG;
  int64_t nb = nblocks(n, block);
  int status = ZQO_OK;
#pragma omp parallel for schedule(static) reduction(min : status)
  for (int64_t b = 0; b < nb; ++b) {
    float v[ZQO_MAX_BLOCK];
    int q[ZQO_MAX_BLOCK + 1];
    int64_t base = b * block, len = n - base < block ? n - base : block;
    for (int64_t i = 0; i < len; ++i) v[i] = load_elem(g, gt, base + i);
    if (quantize_block(v, len, 7, q, &scales[b]) != ZQO_OK) status = ZQO_E_RANGE;
    q[len] = 0;
    for (int64_t i = 0; i < len; i += 2)
      packed[(base + i) >> 1] = (uint8_t)((q[i] & 0x0f) | ((q[i + 1] & 0x0f) << 4));
  }
  return status;
}

/* qgZ dequantiser: y_i = cvt(fl(nibble_i * scale_b)). */
int zqo_qgz_dequantize(const uint8_t* packed, const float* scales, int64_t n, int32_t block, void* y, int yt) {
  if (n < 0 || !block_ok(block) || !dtype_ok(yt)) return ZQO_E_ARG;
  if (n == 0) return ZQO_OK;
  if (!packed || !scales || !y) return ZQO_E_ARG;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    float prod = (float)nibble_at(packed, i) * scales[i / block];
    store_elem(y, yt, i, prod);
  }
  return ZQO_OK;
}

/* qgZ receiver step of the all-to-all reduce-scatter: P INT4 slices of m
 * elements each (slice p at packed_in + p*ceil(m/2) bytes, its scales at
 * scales_in + p*ceil(m/B)) are dequantised, summed and quantised again:
 *   acc_i = +0;  for p = 0 .. P-1:  acc_i = fl(acc_i + fl(q^p_i * s^p_b))
 *   (packed_out, scales_out) = INT4 block quantisation of acc. */
int zqo_qgz_reduce_level(const uint8_t* packed_in, const float* scales_in, int32_t P, int64_t m,
                         int32_t block, uint8_t* packed_out, float* scales_out) {
  if (m < 0 || P < 1 || !block_ok(block)) return ZQO_E_ARG;
  if (m == 0) return ZQO_OK;
  if (!packed_in || !scales_in || !packed_out || !scales_out) return ZQO_E_ARG;
  int64_t slice_bytes = (m + 1) / 2, nb = nblocks(m, block);
  int status = ZQO_OK;
#pragma omp parallel for schedule(static) reduction(min : status)
  for (int64_t b = 0; b < nb; ++b) {
    float acc[ZQO_MAX_BLOCK];
    int q[ZQO_MAX_BLOCK + 1];
    int64_t base = b * block, len = m - base < block ? m - base : block;
    for (int64_t i = 0; i < len; ++i) {
      float sum = 0.0f;
      for (int32_t p = 0; p < P; ++p) {
        float prod = (float)nibble_at(packed_in + (int64_t)p * slice_bytes, base + i) *
                     scales_in[(int64_t)p * nb + b];
        sum = sum + prod;
      }
      acc[i] = sum;
    }
    if (quantize_block(acc, len, 7, q, &scales_out[b]) != ZQO_OK) status = ZQO_E_RANGE;
    q[len] = 0;
    for (int64_t i = 0; i < len; i += 2)
      packed_out[(base + i) >> 1] = (uint8_t)((q[i] & 0x0f) | ((q[i + 1] & 0x0f) << 4));
  }
  return status;
}

/* Format helpers, exposed so tests can pin them against library conversions. */
uint16_t zqo_f32_to_f16(float f) { return f32_to_f16(f); }
uint16_t zqo_f32_to_bf16(float f) { return f32_to_bf16(f); }
float zqo_f16_to_f32(uint16_t h) { return f16_to_f32(h); }
