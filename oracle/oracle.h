/*
 * oracle.h -- CPU oracle for the Auto-Precision-Scaling (APS) gradient path.
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke
 * check and the CPU-baseline leg of the benchmark may load this library.
 * It shares no code, header, table or constant with the HIP library.
 *
 * Every routine works on host arrays, in plain scalar code, with all
 * rounding done exactly in double precision (frexp / ldexp / nearbyint),
 * following Han, Demmel & You, "Auto-Precision Scaling for Distributed Deep
 * Learning" (arXiv 1911.08907):
 *   - Algorithm 1 (APS) for the order of the steps,
 *   - Sec. 3.3.3, Eq. (1)-(4) and the assignment that follows them, for the
 *     per-layer power-of-two scale,
 *   - Sec. 4 (round-to-nearest-even casting) and Table 2 (format ranges) for
 *     the custom float format,
 *   - Sec. 5 (CPD) for the low-precision accumulator of the SUM all-reduce.
 *
 * Readings where the paper is silent are listed at each function.
 */
#ifndef APS_ORACLE_H
#define APS_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A custom float: 1 sign bit, e exponent bits, m mantissa bits, exponent
 * bias.  Algorithm 1 names only exp_bit and man_bit; the bias defaults to
 * 2^(e-1)-1, which is Algorithm 1's upper_bound_exp. */
typedef struct {
    int32_t e;
    int32_t m;
    int32_t bias;
} oracle_format;

/* flags of oracle_sim_reduce */
#define ORACLE_INPUT_QUANTIZED 1u /* input already scaled: skip the 2^f multiply */
#define ORACLE_OUTPUT_SCALED 2u   /* skip the final division by 2^f          */

/* 1 if the format is inside the range this oracle models (e in [2,8],
 * m in [0,23], largest exponent <= 127, smallest subnormal >= 2^-149). */
int oracle_format_ok(oracle_format f);
int oracle_emin(oracle_format f);
int oracle_emax(oracle_format f);
double oracle_maxfinite(oracle_format f);
double oracle_minsub(oracle_format f);

/* The cast of Algorithm 1, R(y): round-to-nearest-even of the real value y
 * to the format; result returned as a double that holds the format value. */
double oracle_round(double y, oracle_format f);

/* Exact ceil(log2 t) for finite t > 0. */
int oracle_ceil_log2(double t);

/* Sec. 3.3.3's exponent of the tensor N * g taken element by element, the
 * route Algorithm 1 describes: the largest ceil(log2|v|) over the nonzero
 * finite products v = fl32(N * g[k]), k < cnt.  Returns INT32_MIN when there
 * is none.  *nonfinite is set to 1 when some product is INF or NaN. */
int32_t oracle_find_max_exp(const float* g, int64_t cnt, int32_t N, int32_t* nonfinite);

/* Per-layer max |G[w][j]| over all W workers and all j of the layer, as the
 * fp32 bit pattern of the magnitude (NaN above INF above every finite). */
void oracle_layer_maxabs(const float* G, int32_t W, int64_t ld, int64_t n,
                         const int64_t* offsets, int32_t L, uint32_t* maxabs_bits);

/* Per-layer scale exponent f = emax - ceil(log2 fl32(N * ghat)). */
int32_t oracle_scale_one(uint32_t maxabs_bits, int32_t N, oracle_format f);
void oracle_layer_scales(const uint32_t* maxabs_bits, int32_t L, int32_t N,
                         const oracle_format* fmts, const uint8_t* fmt_idx,
                         int32_t* scale_exp);

/* Q[w][j] = R(fl32(X[w][j] * 2^f_i)) for j in layer i (scale_exp NULL
 * means f_i = 0 for every layer). */
void oracle_quantize(const float* X, int32_t W, int64_t ld, int64_t n,
                     const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                     const oracle_format* fmts, const uint8_t* fmt_idx, float* Q);

/* Scale, cast, W-worker sum in worker order 0..W-1 with the accumulator
 * rounded to the format after every add, cast back, unscale. */
void oracle_sim_reduce(const float* G, int32_t W, int64_t ld, int64_t n,
                       const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                       const oracle_format* fmts, const uint8_t* fmt_idx,
                       uint32_t flags, float* out);

/* out[j] = fl32(V[j] / 2^f_i) where V is either Q (fp32 values) or the
 * decoded codes. */
void oracle_dequantize(const float* Q, const void* codes, int64_t n,
                       const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                       const oracle_format* fmts, const uint8_t* fmt_idx, float* out);

/* Bit codes: sign << (e+m) | biased exponent << m | mantissa. */
uint32_t oracle_encode(double v, oracle_format f); /* v must be a format value, INF or NaN */
double oracle_decode(uint32_t code, oracle_format f);

/* Pack the format values V[0..n) (each layer with its own format) into codes:
 * 1..4-bit codes two per byte (element 2i in the low nibble of byte i),
 * 5..8-bit codes one byte each, 9..16-bit codes one little-endian uint16. */
void oracle_pack_codes(const float* V, int64_t n, const int64_t* offsets, int32_t L,
                       const oracle_format* fmts, const uint8_t* fmt_idx, void* codes);

/* The SUM all-reduce of Algorithm 1 applied to the cast gradients as the
 * workers would exchange them: W rows of packed codes (row stride ld
 * elements, code layout as in oracle_pack_codes), already scaled and cast.
 * Per element: s = decode(c_0); s = R(s + decode(c_w)) for w = 1..W-1;
 * out = s / 2^ft
 * (or s with ORACLE_OUTPUT_SCALED). */
void oracle_sim_reduce_codes(const void* codes, int32_t W, int64_t ld, int64_t n,
                             const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                             const oracle_format* fmts, const uint8_t* fmt_idx,
                             uint32_t flags, float* out);

/* Accumulation strategies of Sec. 5 (CPD) for a chain of adds. */
#define ORACLE_ACC_SEQUENTIAL 0 /* s = R(s + x) */
#define ORACLE_ACC_KAHAN 1      /* Kahan's compensated summation, every op cast */

/* The SUM all-reduce with the summation order of Sec. 4.2's hierarchical
 * all-reduce and a chosen accumulation strategy.  The W workers form W/k
 * groups of k consecutive workers; a group's master (its first worker) sums
 * the group in worker order; the masters then run a ring reduce-scatter, so
 * segment s of the gradient (element j belongs to s = floor(j * (W/k) / n))
 * accumulates the group sums in master order s, s+1, ..., s+W/k-1 (mod W/k).
 * k = W is the plain worker order 0..W-1, k = 1 a ring over all workers. */
void oracle_sim_reduce_ex(const float* G, int32_t W, int64_t ld, int64_t n,
                          const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                          const oracle_format* fmts, const uint8_t* fmt_idx,
                          uint32_t flags, int32_t group, int32_t accumulator, float* out);

/* Sec. 5 (CPD): C[M][N] = A[M][K] * B[K][N] (row-major, leading dimensions
 * lda, ldb, ldc) on a low-precision multiply-accumulate unit: inputs cast to
 * `in`, every product cast to `acc`, the K products of an output summed in k
 * order by a chain of adds in `acc` (ORACLE_ACC_SEQUENTIAL or
 * ORACLE_ACC_KAHAN), every intermediate cast.  C holds the format values;
 * K = 0 gives +0. */
void oracle_lp_gemm(const float* A, int64_t lda, const float* B, int64_t ldb, float* C, int64_t ldc,
                    int32_t M, int32_t N, int32_t K, oracle_format in, oracle_format acc,
                    int32_t accumulator);

/* Eq. (5) of Sec. 4.2: the mean over the elements with grad_h != 0 of
 * |(grad_h - grad_l) / grad_h|; elements with grad_h == 0 are left out. */
double oracle_round_off_error(const float* grad_h, const float* grad_l, int64_t n);

#ifdef __cplusplus
}
#endif
#endif
