/*
 * abi_check.c -- a plain C (C11) consumer of include/zq.h.  Test
 * infrastructure: it links libzq.so and the CPU oracle (oracle/zq_oracle.c),
 * runs every entry point on device buffers it allocates with the HIP runtime,
 * and compares the results with the oracle's, byte for byte (the GEMM on
 * inputs whose every partial sum is exact, so it too must match exactly).
 * Exit status 0 when everything matches, 1 otherwise.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "zq.h"

/* the CPU oracle (oracle/zq_oracle.c) */
int zqo_qwz_quantize(const void* x, int xt, int64_t n, int32_t block, int8_t* codes, float* scales);
int zqo_qwz_dequantize(const int8_t* codes, const float* scales, int64_t n, int32_t block, void* y, int yt);
int zqo_qgz_quantize(const void* g, int gt, int64_t n, int32_t block, uint8_t* packed, float* scales);
int zqo_qgz_dequantize(const uint8_t* packed, const float* scales, int64_t n, int32_t block, void* y, int yt);
int zqo_qgz_reduce_level(const uint8_t* packed_in, const float* scales_in, int32_t P, int64_t m, int32_t block,
                         uint8_t* packed_out, float* scales_out);

static int failures = 0;

#define HIP_OK(call)                                                            \
  do {                                                                          \
    hipError_t e_ = (call);                                                     \
    if (e_ != hipSuccess) {                                                     \
      fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #call, hipGetErrorString(e_)); \
      exit(2);                                                                  \
    }                                                                           \
  } while (0)

static void expect_status(int got, int want, const char* what) {
  if (got != want) {
    fprintf(stderr, "%s: status %d (%s), want %d\n", what, got, zq_status_string(got), want);
    ++failures;
  }
}

/* device buffer of `bytes`, filled with 0xA5 so an unwritten byte shows */
static void* dev_alloc(size_t bytes) {
  void* p = NULL;
  HIP_OK(hipMalloc(&p, bytes ? bytes : 1));
  HIP_OK(hipMemset(p, 0xA5, bytes ? bytes : 1));
  return p;
}

static void* to_dev(const void* h, size_t bytes) {
  void* d = dev_alloc(bytes);
  HIP_OK(hipMemcpy(d, h, bytes, hipMemcpyHostToDevice));
  return d;
}

static void compare(const void* dev, const void* want, size_t bytes, const char* what) {
  unsigned char* got = malloc(bytes ? bytes : 1);
  HIP_OK(hipMemcpy(got, dev, bytes, hipMemcpyDeviceToHost));
  if (memcmp(got, want, bytes) != 0) {
    size_t i = 0;
    while (i < bytes && got[i] == ((const unsigned char*)want)[i]) ++i;
    fprintf(stderr, "%s: differs from the oracle at byte %zu of %zu\n", what, i, bytes);
    ++failures;
  }
  free(got);
}

/* xorshift64*: deterministic synthetic inputs */
static uint64_t rng = 0x9E3779B97F4A7C15ull;
static double uniform01(void) {
  rng ^= rng >> 12;
  rng ^= rng << 25;
  rng ^= rng >> 27;
  return (double)((rng * 0x2545F4914F6CDD1Dull) >> 11) * (1.0 / 9007199254740992.0);
}
static float gauss(float sd) {
  double u = uniform01(), v = uniform01();
  return (float)(sd * sqrt(-2.0 * log(u + 1e-300)) * cos(6.283185307179586 * v));
}

static int64_t nscales(int64_t n, int32_t b) { return (n + b - 1) / b; }

int main(void) {
  hipStream_t st;
  HIP_OK(hipStreamCreate(&st));

  /* qwZ: fp32 weights, ragged n, INT8 B = 256, dequantised to fp32 */
  {
    const int64_t n = 3 * 1024 * 1024 + 777;
    const int32_t B = 256;
    float* x = malloc(n * sizeof(float));
    for (int64_t i = 0; i < n; ++i) x[i] = gauss(0.02f);
    int8_t* oc = malloc(n);
    float* os = malloc(nscales(n, B) * sizeof(float));
    float* oy = malloc(n * sizeof(float));
    zqo_qwz_quantize(x, ZQ_F32, n, B, oc, os);
    zqo_qwz_dequantize(oc, os, n, B, oy, ZQ_F32);
    void* dx = to_dev(x, n * sizeof(float));
    int8_t* dc = dev_alloc(n);
    float* ds = dev_alloc(nscales(n, B) * sizeof(float));
    float* dy = dev_alloc(n * sizeof(float));
    expect_status(qwz_quantize(dx, ZQ_F32, n, B, dc, ds, st), ZQ_OK, "qwz_quantize");
    expect_status(qwz_dequantize(dc, ds, n, B, dy, ZQ_F32, st), ZQ_OK, "qwz_dequantize");
    HIP_OK(hipStreamSynchronize(st));
    compare(dc, oc, n, "qwz codes");
    compare(ds, os, nscales(n, B) * sizeof(float), "qwz scales");
    compare(dy, oy, n * sizeof(float), "qwz dequant");
    /* an argument error writes nothing and names itself */
    expect_status(qwz_quantize(dx, ZQ_F32, n, 48, dc, ds, st), ZQ_E_BLOCK, "qwz_quantize block 48");
    HIP_OK(hipFree(dx)); HIP_OK(hipFree(dc)); HIP_OK(hipFree(ds)); HIP_OK(hipFree(dy));
    free(x); free(oc); free(os); free(oy);
  }

  /* qgZ: three fp32 gradient slices, INT4 B = 128, one reduce level, the
     final dequantisation, and the fused last level */
  {
    const int32_t P = 3, B = 128;
    const int64_t m = 1 << 20, mb = m / 2, ms = nscales(m, B);
    uint8_t* pin = malloc(P * mb);
    float* sin_ = malloc(P * ms * sizeof(float));
    float* g = malloc(m * sizeof(float));
    for (int p = 0; p < P; ++p) {
      for (int64_t i = 0; i < m; ++i) g[i] = gauss(p == 1 ? 1e-2f : 1e-3f);
      zqo_qgz_quantize(g, ZQ_F32, m, B, pin + p * mb, sin_ + p * ms);
    }
    uint8_t* orp = malloc(mb);
    float* ors = malloc(ms * sizeof(float));
    float* oy = malloc(m * sizeof(float));
    zqo_qgz_reduce_level(pin, sin_, P, m, B, orp, ors);
    zqo_qgz_dequantize(orp, ors, m, B, oy, ZQ_F32);
    /* the quantiser itself, on the last slice's source */
    uint8_t* oq = malloc(mb);
    float* oqs = malloc(ms * sizeof(float));
    zqo_qgz_quantize(g, ZQ_F32, m, B, oq, oqs);
    void* dg = to_dev(g, m * sizeof(float));
    uint8_t* dq = dev_alloc(mb);
    float* dqs = dev_alloc(ms * sizeof(float));
    expect_status(qgz_quantize(dg, ZQ_F32, m, B, dq, dqs, st), ZQ_OK, "qgz_quantize");
    uint8_t* dpin = to_dev(pin, P * mb);
    float* dsin = to_dev(sin_, P * ms * sizeof(float));
    uint8_t* drp = dev_alloc(mb);
    float* drs = dev_alloc(ms * sizeof(float));
    float* dy = dev_alloc(m * sizeof(float));
    float* dyf = dev_alloc(m * sizeof(float));
    expect_status(qgz_reduce_level(dpin, dsin, P, m, B, drp, drs, st), ZQ_OK, "qgz_reduce_level");
    expect_status(qgz_dequantize(drp, drs, m, B, dy, ZQ_F32, st), ZQ_OK, "qgz_dequantize");
    expect_status(qgz_reduce_dequantize(dpin, dsin, P, m, B, dyf, ZQ_F32, NULL, NULL, st), ZQ_OK,
                  "qgz_reduce_dequantize");
    HIP_OK(hipStreamSynchronize(st));
    compare(dq, oq, mb, "qgz packed");
    compare(dqs, oqs, ms * sizeof(float), "qgz scales");
    compare(drp, orp, mb, "reduce packed");
    compare(drs, ors, ms * sizeof(float), "reduce scales");
    compare(dy, oy, m * sizeof(float), "final dequant");
    compare(dyf, oy, m * sizeof(float), "fused last level");
    expect_status(qgz_reduce_level(dpin, dsin, 0, m, B, drp, drs, st), ZQ_E_P, "reduce P = 0");
    /* the same level through device tables of slice pointers */
    {
      const uint8_t* hp[3];
      const float* hs[3];
      for (int p = 0; p < P; ++p) {
        hp[p] = dpin + p * mb;
        hs[p] = dsin + p * ms;
      }
      const uint8_t** tp = to_dev(hp, sizeof hp);
      const float** ts = to_dev(hs, sizeof hs);
      uint8_t* grp = dev_alloc(mb);
      float* grs = dev_alloc(ms * sizeof(float));
      expect_status(qgz_reduce_level_gather(tp, ts, P, m, B, grp, grs, st), ZQ_OK, "qgz_reduce_level_gather");
      HIP_OK(hipStreamSynchronize(st));
      compare(grp, orp, mb, "gather packed");
      compare(grs, ors, ms * sizeof(float), "gather scales");
      /* the allocation-free form: the same addresses from host arrays */
      HIP_OK(hipMemset(grp, 0xA5, mb));
      HIP_OK(hipMemset(grs, 0xA5, ms * sizeof(float)));
      expect_status(qgz_reduce_level_gather_noalloc(hp, hs, P, m, B, grp, grs, st), ZQ_OK,
                    "qgz_reduce_level_gather_noalloc");
      HIP_OK(hipStreamSynchronize(st));
      compare(grp, orp, mb, "gather (no alloc) packed");
      compare(grs, ors, ms * sizeof(float), "gather (no alloc) scales");
      expect_status(qgz_reduce_level_gather_noalloc(hp, hs, 1025, m, B, grp, grs, st), ZQ_E_P, "no-alloc P = 1025");
      HIP_OK(hipFree((void*)tp)); HIP_OK(hipFree((void*)ts)); HIP_OK(hipFree(grp)); HIP_OK(hipFree(grs));
    }
    HIP_OK(hipFree(dg)); HIP_OK(hipFree(dq)); HIP_OK(hipFree(dqs)); HIP_OK(hipFree(dpin)); HIP_OK(hipFree(dsin));
    HIP_OK(hipFree(drp)); HIP_OK(hipFree(drs)); HIP_OK(hipFree(dy)); HIP_OK(hipFree(dyf));
    free(pin); free(sin_); free(g); free(orp); free(ors); free(oy); free(oq); free(oqs);
  }

  /* dequantise-on-load GEMM: bf16 x in multiples of 1/4, scales 2^-7, so the
     product is exact in any summation order */
  {
    const int64_t M = 100, N = 192, K = 256;
    const int32_t B = 64;
    uint16_t* x = malloc(M * K * sizeof(uint16_t));
    for (int64_t i = 0; i < M * K; ++i) {
      float v = (float)((int)(uniform01() * 33.0) - 16) * 0.25f;
      uint32_t u;
      memcpy(&u, &v, 4);
      x[i] = (uint16_t)(u >> 16); /* exact: v has at most 6 significant bits */
    }
    int8_t* c = malloc(N * K);
    for (int64_t i = 0; i < N * K; ++i) c[i] = (int8_t)((int)(uniform01() * 255.0) - 127);
    float* s = malloc(nscales(N * K, B) * sizeof(float));
    for (int64_t i = 0; i < nscales(N * K, B); ++i) s[i] = 1.0f / 128.0f;
    uint16_t* w = malloc(N * K * sizeof(uint16_t));
    zqo_qwz_dequantize(c, s, N * K, B, w, ZQ_BF16);
    float* want = malloc(M * N * sizeof(float));
    for (int64_t i = 0; i < M; ++i)
      for (int64_t j = 0; j < N; ++j) {
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k) {
          uint32_t ux = (uint32_t)x[i * K + k] << 16, uw = (uint32_t)w[j * K + k] << 16;
          float fx, fw;
          memcpy(&fx, &ux, 4);
          memcpy(&fw, &uw, 4);
          acc += (double)fx * (double)fw;
        }
        want[i * N + j] = (float)acc;
      }
    void* dx = to_dev(x, M * K * sizeof(uint16_t));
    int8_t* dc = to_dev(c, N * K);
    float* ds = to_dev(s, nscales(N * K, B) * sizeof(float));
    float* dy = dev_alloc(M * N * sizeof(float));
    expect_status(qwz_dequant_gemm(dx, ZQ_BF16, dc, ds, M, N, K, B, dy, st), ZQ_OK, "qwz_dequant_gemm");
    HIP_OK(hipStreamSynchronize(st));
    compare(dy, want, M * N * sizeof(float), "dequantise GEMM");
    expect_status(qwz_dequant_gemm(dx, ZQ_BF16, dc, ds, M, N, 96, B, dy, st), ZQ_E_SIZE, "GEMM K = 96");
    HIP_OK(hipFree(dx)); HIP_OK(hipFree(dc)); HIP_OK(hipFree(ds)); HIP_OK(hipFree(dy));
    free(x); free(c); free(s); free(w); free(want);
  }

  if (zq_num_scales(123456789, 64) != 1929013 || zq_int4_bytes(123456789) != 61728395) {
    fprintf(stderr, "size helpers\n");
    ++failures;
  }
  HIP_OK(hipStreamDestroy(st));
  if (failures) {
    fprintf(stderr, "abi_check: %d failure(s)\n", failures);
    return 1;
  }
  printf("abi_check ok\n");
  return 0;
}
