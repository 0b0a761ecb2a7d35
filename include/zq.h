/*
 * zq.h -- C ABI of the qwZ / qgZ compression data path for one MI355X (gfx950).
 *
 * Method: arXiv 2501.04266 ("Scaling Large Language Model Training on
 * Frontier with Low-Bandwidth Partitioning").  Its hierarchical ZeRO++
 * partitioning compresses every collective with ZeRO++'s block-based
 * quantisation (Background, ZeRO++ subsection): weights are quantised to
 * INT8 blocks before the weight Allgather and dequantised after it (qwZ;
 * Design, Weight Partitioning: quantiser / dequantiser operators, secondary
 * partition stored quantised), and gradients travel as INT4 blocks through an
 * all-to-all reduce-scatter whose receiver dequantises, sums and requantises
 * the P slices it gets (qgZ; Design, Gradient Partitioning and Communication
 * Volume Analysis).  Each block has its own scale (Evaluations, Model
 * Convergence).  This library is one rank's share of that path, with the P
 * slices of a level already resident in this GPU's memory.
 *
 * Definition implemented (symmetric absmax; the paper gives no formula, these
 * are the readings taken):
 *   block b = elements [b*B, min(n, (b+1)*B)); the last block may be short.
 *   a = max |x_i| over the block;   qmax = 127 (INT8) or 7 (INT4)
 *   a < 2^-119 (incl. all-zero):    scale = +0, every code 0
 *   otherwise: scale = fl(a / qmax), r = fl(qmax / a),
 *              code_i = round-half-even(fl(x_i * r))  (always within +-qmax)
 *   dequant:   y_i = cvt(fl(code_i * scale)), cvt = identity or RNE narrowing
 *   reduce:    acc_i = +0; for p = 0..P-1: acc_i = fl(acc_i + fl(q^p_i * s^p_b))
 *              then INT4-quantise acc (one rounded multiply, then one rounded
 *              add per slice; no fused multiply-add).
 * fl() is one IEEE binary32 operation rounded to nearest even; fp32
 * subnormals are kept.  Results are bit-identical to that definition.
 *
 * Formats:
 *   INT8 codes:  int8_t[n], two's complement.
 *   INT4 codes:  uint8_t[ceil(n/2)]; element 2j in the low nibble of byte j,
 *                element 2j+1 in the high nibble, two's complement; for odd n
 *                the last high nibble is 0.
 *   scales:      float[ceil(n/B)], one per block.
 *   elements:    ZQ_F32 (float), ZQ_F16 (IEEE binary16), ZQ_BF16 (bfloat16).
 *
 * Conventions for every call:
 *   - All array pointers are device pointers (hipMalloc'd or equivalent) in
 *     the caller's ownership; the library allocates nothing and keeps no
 *     state between calls, except the device address table of
 *     qgz_reduce_level_gather_noalloc (a static array per GPU).
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the default stream)
 *     and returns without synchronising; results are visible after the
 *     stream is synchronised.  Calls from several host threads are safe.
 *   - block must be a power of two in [32, 1024].
 *   - Element and code arrays must be 16-byte aligned, scale arrays 4-byte
 *     aligned.  Outputs must not overlap inputs.
 *   - n == 0 (or m == 0) is a successful no-op; n < 0 is ZQ_E_SIZE.
 *   - Inputs are expected to be finite; non-finite inputs give unspecified
 *     codes (no error is raised, to avoid an extra pass).
 *   - Every argument error is detected on the host before anything is
 *     enqueued, so no output byte is written.  ZQ_E_HIP means a HIP launch
 *     failed (outputs then undefined).
 */
#ifndef ZQ_H
#define ZQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int zq_dtype;
enum { ZQ_F32 = 0, ZQ_F16 = 1, ZQ_BF16 = 2 };

enum {
  ZQ_OK = 0,
  ZQ_E_NULL = -1,   /* a required pointer is NULL (with n > 0) */
  ZQ_E_BLOCK = -2,  /* block not a power of two in [32, 1024] */
  ZQ_E_DTYPE = -3,  /* unknown element dtype */
  ZQ_E_ALIGN = -4,  /* misaligned pointer */
  ZQ_E_SIZE = -5,   /* negative element count */
  ZQ_E_P = -6,      /* slice count outside [1, 1024] */
  ZQ_E_HIP = -7,    /* HIP kernel launch failed */
  ZQ_E_ALIAS = -8   /* an output overlaps an input */
};

/* qwZ quantiser (Background, ZeRO++: quantise the weight shard to INT8 blocks
 * before the Allgather; Design, Weight Partitioning: also the quantised
 * secondary partition).
 *   x       [n] elements of dtype xt (read)
 *   codes   [n] int8 codes (written)
 *   scales  [ceil(n/block)] floats (written) */
int qwz_quantize(const void* x, zq_dtype xt, int64_t n, int32_t block,
                 int8_t* codes, float* scales, void* stream);

/* qwZ dequantiser (Design, Weight Partitioning: dequantise the gathered layer
 * for the forward pass, or the gathered secondary partition for backward).
 *   codes [n], scales [ceil(n/block)] (read) -> y [n] of dtype yt (written) */
int qwz_dequantize(const int8_t* codes, const float* scales, int64_t n, int32_t block,
                   void* y, zq_dtype yt, void* stream);

/* qgZ quantiser (Background, ZeRO++: gradients quantised to INT4 blocks for
 * the all-to-all reduce-scatter).
 *   g [n] of dtype gt (read) -> packed [ceil(n/2)] bytes, scales [ceil(n/block)] */
int qgz_quantize(const void* g, zq_dtype gt, int64_t n, int32_t block,
                 uint8_t* packed, float* scales, void* stream);

/* qgZ reduce level: the receiver side of the quantised all-to-all
 * reduce-scatter (Background, ZeRO++; Design, Communication Volume Analysis:
 * 1-hop all-to-all within the node).  P slices of m elements each, laid out
 * back to back: slice p's bytes at packed_in + p*ceil(m/2), its scales at
 * scales_in + p*ceil(m/block).  They are dequantised, summed in ascending
 * slice order and requantised to one INT4 slice of m elements:
 *   packed_out [ceil(m/2)], scales_out [ceil(m/block)] (written).
 * 1 <= P <= 1024.  The hierarchical scheme applies this once per partition
 * level (Design: GCD pair, node, all ranks). */
int qgz_reduce_level(const uint8_t* packed_in, const float* scales_in, int32_t P, int64_t m,
                     int32_t block, uint8_t* packed_out, float* scales_out, void* stream);

/* qgZ dequantiser: final gradient shard for the optimizer (Design, Gradient
 * Partitioning).  packed [ceil(n/2)], scales [ceil(n/block)] -> y [n] of yt. */
int qgz_dequantize(const uint8_t* packed, const float* scales, int64_t n, int32_t block,
                   void* y, zq_dtype yt, void* stream);

/* Fused last level: the receiver's final reduce level followed by the
 * dequantisation of the resulting gradient shard for the optimizer (Design,
 * Gradient Partitioning; Background, ZeRO++: quantised reduce-scatter).
 * Writes y [m] of dtype yt, bit-identical to qgz_dequantize applied to what
 * qgz_reduce_level would produce from the same slices, without storing and
 * re-reading the INT4 result.  packed_out / scales_out are optional: both NULL,
 * or both given to receive that INT4 result as well.  Slice layout, limits
 * and errors as qgz_reduce_level; y must be 16-byte aligned and overlap no
 * input or output. */
int qgz_reduce_dequantize(const uint8_t* packed_in, const float* scales_in, int32_t P, int64_t m, int32_t block,
                          void* y, zq_dtype yt, uint8_t* packed_out, float* scales_out, void* stream);

/* Reduce level over slices that are not back to back: the receiver reading
 * each peer's INT4 chunk where it lies, without first copying the chunks into
 * one receive buffer (the peer-direct form of the quantised all-to-all
 * reduce-scatter; Background, ZeRO++; Design, Communication Volume Analysis).
 * On one GPU the slices are separate device buffers; on a node they can be
 * the peers' buffers mapped into this GPU's address space.
 *   packed_slices  device array of P pointers; slice p holds ceil(m/2) bytes
 *   scale_slices   device array of P pointers; slice p holds ceil(m/block) floats
 * Same arithmetic, order and output as qgz_reduce_level on the slices laid
 * out back to back (bit-identical).  The two pointer arrays must be 8-byte
 * aligned and stay unchanged until the call completes; when m % 32 == 0 each
 * byte slice must be 16-byte aligned and each scale slice 4-byte aligned.
 * The library cannot read the device-resident pointers on the host, so only
 * the arrays themselves are checked against the outputs for overlap; the
 * slices must not overlap the outputs either.  Other conventions and errors
 * as qgz_reduce_level. */
int qgz_reduce_level_gather(const uint8_t* const* packed_slices, const float* const* scale_slices, int32_t P,
                            int64_t m, int32_t block, uint8_t* packed_out, float* scales_out, void* stream);

/* Allocation-free form of qgz_reduce_level_gather, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The P slice addresses come in HOST
 * arrays; the library writes them into a static device table of its own (one
 * per GPU, 2048 addresses = 16 KiB, held until the process ends) with small
 * kernels on `stream` whose values travel as kernel arguments, then runs the
 * gathered reduce over them.  Nothing is allocated and nothing synchronises.
 *   packed_slices  host array of P device pointers; slice p holds ceil(m/2) bytes
 *   scale_slices   host array of P device pointers; slice p holds ceil(m/block) floats
 *   packed_out, scales_out as qgz_reduce_level (both required)
 * The host arrays are read before the call returns.  1 <= P <= 1024 (larger P
 * is ZQ_E_P: the table holds 1024 pairs).  Because the addresses are on the
 * host, every slice is checked: non-null (ZQ_E_NULL), 16-byte aligned when
 * m % 32 == 0 and scale slices 4-byte aligned (ZQ_E_ALIGN), no overlap with
 * an output (ZQ_E_ALIAS).  The table belongs to the current device, and
 * `stream` must belong to it too.  Every call on one GPU uses the same table:
 * calls that can overlap on one GPU (different streams, or different host
 * threads without ordering) race on it; calls on one stream are ordered.
 * Results are bit-identical to qgz_reduce_level_gather (and qgz_reduce_level
 * on the slices back to back). */
int qgz_reduce_level_gather_noalloc(const uint8_t* const* packed_slices, const float* const* scale_slices, int32_t P,
                                    int64_t m, int32_t block, uint8_t* packed_out, float* scales_out, void* stream);

/* Dequantise-on-load GEMM: the forward product of a layer whose weight
 * arrives as the gathered INT8 buffer (Design, Weight Partitioning: the
 * Allgathered weights are dequantised for the forward pass), without writing
 * the dequantised weight to memory:
 *   y[m][n] = sum_k x[m][k] * w[n][k],  w[n][k] = cvt(fl(q[n*K + k] * s[(n*K + k) / block]))
 * i.e. w is exactly what qwz_dequantize(codes, scales, N*K, block, ., xt)
 * writes, and the sum is taken in binary32 by the matrix cores in an order of
 * their own, always within 2*K*2^-24 * sum_k |x[m][k] w[n][k]| of the exact
 * value.  When the output tiles alone would leave much of the GPU idle (few
 * rows, or a few hundred rows with few tiles), the K range may be split across
 * workgroups whose partial sums are added into y atomically (after the
 * library zeroes y), so such results can differ between runs in their last
 * bits.
 *   x       [M][K] row-major, xt = ZQ_BF16 or ZQ_F16 (read)
 *   codes   [N][K] int8 row-major (a PyTorch Linear weight, flattened), scales
 *           [ceil(N*K/block)] floats (read)
 *   y       [M][N] float row-major (written)
 * K must be a multiple of 64 (ZQ_E_SIZE otherwise); M, N >= 0 arbitrary; K = 0
 * writes zeros.  x and codes 16-byte aligned, scales and y 4-byte aligned; y
 * must not overlap an input.  Other conventions as above.
 * When to use it: on MI355X this call is faster than qwz_dequantize of the
 * layer followed by a library bf16 GEMM (hipBLASLt) up to about 1,000 rows of
 * x (GPT-20B layer's four GEMMs: 0.15 against 0.53 ms at 16 rows, 0.22 against
 * 0.53 ms at 64, about 1.05 against 1.15 ms at 1,024).  With many more rows
 * the separate path wins (6.1 against 5.2 ms at 8,192), so large batches
 * should dequantise the gathered layer once and call a library GEMM. */
int qwz_dequant_gemm(const void* x, zq_dtype xt, const int8_t* codes, const float* scales, int64_t M, int64_t N,
                     int64_t K, int32_t block, float* y, void* stream);

/* Size helpers (host only): number of scales ceil(n/block) (-1 on a bad
 * block or n < 0), and INT4 bytes ceil(n/2) (-1 for n < 0). */
int64_t zq_num_scales(int64_t n, int32_t block);
int64_t zq_int4_bytes(int64_t n);

/* Static, human-readable name of a status code. */
const char* zq_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* ZQ_H */
