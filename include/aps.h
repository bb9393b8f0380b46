/*
 * aps.h -- C ABI of the MI355X (gfx950) Auto-Precision-Scaling gradient path.
 *
 * Paper: Han, Demmel, You, "Auto-Precision Scaling for Distributed Deep
 * Learning", arXiv 1911.08907.  The five compute calls are the steps of
 * Algorithm 1 (APS) for one synchronisation of a model's gradients, with the
 * W data-parallel workers simulated on one GPU:
 *
 *   aps_layer_maxabs   FindMaxExp input + AllReduce(MAX)   (Alg. 1, FindMaxExp)
 *   aps_layer_scales   ft = upper_bound_exp - max exponent (Alg. 1; Sec. 3.3.3)
 *   aps_quantize       scale by 2^ft, cast to the format   (Alg. 1; Sec. 3.3.1)
 *   aps_sim_reduce     scale, cast, AllReduce(SUM) with a low-precision
 *                      accumulator, cast back, unscale     (Alg. 1; Sec. 5)
 *   aps_dequantize     back to fp32, scale undone          (Alg. 1)
 *
 * Beside them, CPD's accumulation experiments (Sec. 5): aps_sim_reduce_ex
 * (summation orders, Kahan), aps_sim_reduce_codes (the sum over packed
 * codes) and aps_lp_gemm (a GEMM with a low-precision accumulator).
 *
 * Data layout.  A model's gradients are one flat fp32 vector of n elements;
 * layer i (one parameter tensor) owns elements [offsets[i], offsets[i+1]).
 * W workers' gradients are stored worker-major: element j of worker w is
 * G[w * ld + j], with row stride ld >= n.
 *
 * Custom float format {e, m, bias}: 1 sign bit, e exponent bits, m mantissa
 * bits.  IEEE-754 layout: exponent field 0 holds zero and the subnormals
 * (value mant * 2^(1-bias-m)), the all-ones field holds INF (mant 0) and NaN.
 * Rounding is round-to-nearest-even; a magnitude at or above
 * (2 - 2^-(m+1)) * 2^emax becomes INF, one at or below half the smallest
 * subnormal becomes a zero of the input's sign.  With m = 0 a tie goes to
 * the even multiple of the quantum (significand 1.1b rounds up to 10b).
 * emin = 1 - bias, emax = 2^e - 2 - bias.  The default bias 2^(e-1)-1 gives
 * Algorithm 1's upper_bound_exp as emax and Table 2's ranges.
 *
 * Memory.  Every array argument except `fmts` is DEVICE memory owned by the
 * caller.  `fmts` is HOST memory, read during the call only.  The calls
 * allocate nothing and keep no state between calls; the one static device
 * array of aps_sync_noalloc (below) is the only memory the library holds.
 *
 * Streams.  `stream` is a hipStream_t (NULL = the default stream).  A call
 * validates its arguments on the host, enqueues its kernels on `stream` and
 * returns without synchronising.  Calls are thread-safe.
 *
 * Errors.  Argument checks happen on the host before anything is enqueued and
 * return a negative status; a failed launch returns APS_ERR_DEVICE.  The
 * contents of device arrays are not checked: offsets must start at 0, be
 * non-decreasing and end at n; every fmt_idx[i] must be < n_fmts.  Other
 * contents give undefined results.
 *
 * Bit codes.  code = sign << (e+m) | biased exponent << m | mantissa.  A NaN
 * is written as the all-ones exponent with the top mantissa bit set (the INF
 * code when m = 0); the sign bit of a NaN's code is unspecified.  Codes of
 * 2..4 bits are packed two per byte (element j in the low nibble of byte j/2
 * when j is even, the high nibble when odd); codes of 5..8 bits take one
 * byte; codes of 9..16 bits one little-endian uint16.
 * A call that writes or reads codes needs every format of its palette in the
 * same one of those three classes.
 */
#ifndef APS_H
#define APS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t e;    /* exponent bits, 2..8 */
    int32_t m;    /* mantissa bits, 0..23 */
    int32_t bias; /* exponent bias; default (1 << (e-1)) - 1 */
} aps_format;

enum {
    APS_OK = 0,
    APS_ERR_NULL = -1,        /* a required pointer is NULL */
    APS_ERR_SIZE = -2,        /* W, L, n, ld, n_fmts or N out of range */
    APS_ERR_FORMAT = -3,      /* e, m or bias outside the supported range */
    APS_ERR_ALIGN = -4,       /* a pointer or ld breaks the alignment rules */
    APS_ERR_UNSUPPORTED = -5, /* valid but not provided (see aps_format_supported) */
    APS_ERR_DEVICE = -6       /* a HIP call or kernel launch failed */
};

/* sim_reduce flags */
#define APS_INPUT_QUANTIZED 1u /* G is already scaled by 2^ft: skip that multiply (the
                                * cast is still applied; it is exact on format values) */
#define APS_OUTPUT_SCALED 2u   /* leave the sum scaled: skip the division by 2^ft */

/* Limits checked on the host. */
#define APS_MAX_FORMATS 8          /* palette size n_fmts is 1..8 */
#define APS_MAX_WORKERS (1 << 24)  /* W and N: N * max|g| is an fp32 product */
#define APS_MAX_ELEMS (1LL << 30)  /* n (elements per worker) */

/*
 * Returns APS_OK if {e, m, bias} is a format the kernels implement, else
 * APS_ERR_FORMAT (outside e in [2,8], m in [0,23], emax <= 127,
 * emin - m >= -149): every format whose values fp32 holds.  Formats with
 * e = 8 and a bias other than 127, or whose half-smallest-subnormal lies
 * below 2^-126, round in fp64 (slower) and are not taken by the one-pass
 * route of aps_sync nor by aps_lp_gemm.  Host-only; never touches the GPU.
 */
int aps_format_supported(aps_format f);

/*
 * Per-layer maximum magnitude over all W workers (Algorithm 1: the input of
 * FindMaxExp and its AllReduce(MAX); the maximum of ceil(log2|N*g|) over a
 * layer is taken from the maximum |g|, since both maps are monotone).
 *
 *   G            [W][ld] fp32, 16-byte aligned, ld % 4 == 0, ld >= n
 *   offsets      int64[L+1] layer boundaries
 *   maxabs_bits  uint32[L] out: fp32 bit pattern of max |G[w][j]| over all
 *                w and all j of the layer; a NaN anywhere gives a NaN
 *                pattern (above 0x7F800000), an empty or all-zero layer 0.
 * Sizes: 1 <= W <= APS_MAX_WORKERS, L >= 1, 0 <= n <= APS_MAX_ELEMS.
 */
int aps_layer_maxabs(const float* G, int32_t W, int64_t ld, int64_t n,
                     const int64_t* offsets, int32_t L, uint32_t* maxabs_bits,
                     void* stream);

/*
 * Per-layer power-of-two scale exponent (Sec. 3.3.3 and Algorithm 1):
 *   scale_exp[i] = emax(fmt_i) - ceil(log2 fl32(N * ghat_i))
 * where ghat_i is the magnitude in maxabs_bits[i] and fl32 the fp32 product.
 * It is the largest exponent with N * ghat_i * 2^scale_exp[i] <= 2^emax.
 * A layer with ghat 0, INF or NaN, or with fl32(N * ghat) = INF, gets 0.
 *
 *   maxabs_bits  uint32[L] (device), e.g. from aps_layer_maxabs
 *   N            number of workers, 1..APS_MAX_WORKERS
 *   fmts         host aps_format[n_fmts], 1 <= n_fmts <= APS_MAX_FORMATS
 *   fmt_idx      uint8[L] (device) palette index per layer, or NULL (all 0)
 *   scale_exp    int32[L] out
 */
int aps_layer_scales(const uint32_t* maxabs_bits, int32_t L, int32_t N,
                     const aps_format* fmts, int32_t n_fmts, const uint8_t* fmt_idx,
                     int32_t* scale_exp, void* stream);

/*
 * Scale and cast every element of every worker (Algorithm 1: the gradient
 * times 2^ft, then the cast to the custom format):
 *   Q[w][j] = R_fmt(fl32(X[w][j] * 2^scale_exp[i]))   for j in layer i.
 * The product is the fp32 value nearest to X * 2^ft; R_fmt is the format's
 * round-to-nearest-even described above.
 *
 *   X          [W][ld] fp32 (16-byte aligned, ld % 4 == 0)
 *   scale_exp  int32[L] or NULL (every ft = 0: casting without APS)
 *   Q          [W][ld] fp32 out, may be X itself; or NULL
 *   codes      [W][ld] packed codes out (row stride ld elements), 16-byte
 *              aligned; or NULL.  At least one of Q, codes is non-NULL.
 * Elements j in [n, ld) of each row are not written.
 */
int aps_quantize(const float* X, int32_t W, int64_t ld, int64_t n,
                 const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                 const aps_format* fmts, int32_t n_fmts, const uint8_t* fmt_idx,
                 float* Q, void* codes, void* stream);

/*
 * The fused APS step for one simulated synchronisation (Algorithm 1 with
 * the low-precision accumulator of Sec. 5), per element j of layer i:
 *   q_w = R_fmt(fl32(G[w][j] * 2^ft))            w = 0..W-1
 *   s   = q_0;  s = R_fmt(s + q_w) for w = 1..W-1   (this order, rounded
 *                                                   after every add)
 *   out[j] = fl32(s / 2^ft)
 * out is the sum over workers (not the mean).  With APS_INPUT_QUANTIZED the
 * multiply by 2^ft is skipped; with APS_OUTPUT_SCALED the division is.
 *
 *   G          [W][ld] fp32 (16-byte aligned, ld % 4 == 0); not aliased by out
 *   scale_exp  int32[L] or NULL (every ft = 0)
 *   out        fp32[n] out (16-byte aligned), or NULL
 *   codes_out  packed codes of the scaled sum s, [n] (16-byte aligned), or NULL
 *   At least one of out, codes_out is non-NULL.
 */
int aps_sim_reduce(const float* G, int32_t W, int64_t ld, int64_t n,
                   const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                   const aps_format* fmts, int32_t n_fmts, const uint8_t* fmt_idx,
                   uint32_t flags, float* out, void* codes_out, void* stream);

/* aps_sync flags: one or both passes, and optionally a route */
#define APS_SYNC_PASS1 1u    /* read G: layer maxima (and, on the one-pass route, the
                              * unscaled rounded sums and the workspace bytes) */
#define APS_SYNC_PASS2 2u    /* scale exponents, then the rest of the sum */
#define APS_SYNC_ONE_PASS 4u /* take the one-pass route wherever it applies */
#define APS_SYNC_TWO_PASS 8u /* always read G twice */
#define APS_SYNC_GUESS 16u   /* take the guessed-scale route */

/* the routes, as aps_sync_route returns them */
#define APS_SYNC_ROUTE_TWO_PASS 0
#define APS_SYNC_ROUTE_ONE_PASS 1
#define APS_SYNC_ROUTE_GUESS 2

/*
 * Bytes of workspace aps_sync needs for n elements and L layers, with
 * C = ceil(n / 1024) chunks: round_up(1024 * C, 256) + round_up(4 * C, 256)
 * + round_up(4 * L, 256) + 256 + round_up(4 * C, 256) + 2048 * C
 * + round_up(4 * L, 256) + round_up(C, 256).  Host-only.
 * Returns 0 for negative arguments or n > APS_MAX_ELEMS.
 */
uint64_t aps_sync_workspace_bytes(int64_t n, int32_t L);

/*
 * Which route aps_sync takes for W workers, n elements, this palette and
 * these flags (only the route bits of flags matter): APS_SYNC_ROUTE_*, or a
 * negative status (W or n out of range, a bad palette, more than one route
 * bit).  Host-only.
 */
int aps_sync_route(int32_t W, int64_t n, const aps_format* fmts, int32_t n_fmts, uint32_t flags);

/*
 * One whole APS synchronisation of W simulated workers (Algorithm 1 with the
 * low-precision accumulator of Sec. 5), with N = W:
 *   maxabs_bits  as aps_layer_maxabs
 *   scale_exp    as aps_layer_scales with N = W
 *   out          as aps_sim_reduce with flags 0 (the unscaled sum)
 * The three arrays hold exactly what those three calls in sequence produce,
 * whichever route is taken.
 *
 * The one-pass route reads G once instead of twice.  Power-of-two scaling
 * commutes with rounding to m+1 significant bits (Sec. 3.3.1), so pass 1
 * forms the rounded sum on the unscaled values while it takes the layer
 * maxima.  Pass 2 computes the scales and recomputes through the scaled
 * path only the elements for which the unscaled sum can differ: those with
 * a nonzero input below T = max(2^(emin - ft), 2^-126) (the format's
 * subnormal range after scaling) that is not swamped, i.e. that comes from
 * worker 0 or meets a partial sum below 2^(m+3) * T, and every element of a
 * layer whose max is INF or NaN or whose N * ghat exceeds 2^127.  Pass 1
 * records one byte per element to find them (with fewer than 64 workers only
 * the minimum byte of each 256-element group, and pass 2 reruns whole
 * groups).  From 128 workers on, with every palette format m <= 7, pass 1
 * keeps each sum in 2 bytes of the workspace (its fp32 pattern's low 16 bits
 * are zero) and pass 2 widens them into out.  The route applies when W is a
 * power of two and every palette format has m <= 10 and rounds in fp32
 * (see aps_format_supported).
 *
 * The guessed-scale route applies to every W and format.  Pass 1 takes the
 * layer maxima of every 32nd worker (rows 0, 32, 64, ...), guesses each
 * layer's scale exponent from them (allowing for the growth of a normal
 * sample's max with the sample size), and then, reading G once, forms the
 * scaled sums with the guesses while it takes the full maxima.  Pass 2
 * computes the true exponents and reruns through the scaled path every
 * chunk of a layer whose guess differs.  The results never depend on the
 * guess; its cost is ceil(W/32) rows read plus the rerun layers.
 *
 * The two-pass route: pass 1 is aps_layer_maxabs, pass 2 aps_layer_scales
 * followed by aps_sim_reduce.
 *
 * Route choice: APS_SYNC_TWO_PASS and APS_SYNC_GUESS force their routes;
 * APS_SYNC_ONE_PASS takes the one-pass route wherever it applies (else two
 * passes).  With no route bit, the one-pass route is taken where it applies
 * and the format's range leaves few elements to recompute
 * (W^2 * 2^(emin - emax + 2) <= 2^-7 for every palette format); otherwise
 * the guessed-scale route when W * n >= 2^26, else two passes.
 *
 *   G          [W][ld] fp32 (16-byte aligned, ld % 4 == 0); not aliased by out
 *   flags      APS_SYNC_PASS1, APS_SYNC_PASS2 or both, plus at most one of
 *              APS_SYNC_ONE_PASS, APS_SYNC_TWO_PASS, APS_SYNC_GUESS.  Run
 *              separately, pass 2 must follow pass 1 with the same arguments
 *              and route flag on the same stream, with the workspace,
 *              scale_exp and out untouched in between; after pass 1 alone,
 *              maxabs_bits is final and scale_exp and out hold intermediate
 *              values
 *   maxabs_bits uint32[L] out
 *   scale_exp  int32[L] out
 *   out        fp32[n] out (16-byte aligned)
 *   workspace  device memory of at least aps_sync_workspace_bytes(n, L)
 *              bytes, 256-byte aligned, owned by the caller; its contents on
 *              entry do not matter
 * Every pass enqueues kernels only (no memset, no allocation, no host
 * synchronisation), so a call can be captured in a HIP graph and replayed.
 * Calls that share a workspace must not overlap.  Errors as aps_sim_reduce;
 * a small workspace returns APS_ERR_SIZE; no pass bit, an unknown bit or more
 * than one route bit return APS_ERR_UNSUPPORTED.
 */
int aps_sync(const float* G, int32_t W, int64_t ld, int64_t n,
             const int64_t* offsets, int32_t L,
             const aps_format* fmts, int32_t n_fmts, const uint8_t* fmt_idx,
             uint32_t flags, uint32_t* maxabs_bits, int32_t* scale_exp, float* out,
             void* workspace, uint64_t workspace_bytes, void* stream);

/*
 * aps_sync for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  It
 * takes no workspace argument; its workspace is a static device array of
 * APS_SYNC_SCRATCH_BYTES bytes that the HIP runtime places on each GPU when
 * it loads this library's code there, and that stays until the process
 * ends.  The call itself allocates nothing: no hipMalloc, no hipFree, no
 * allocating library routine.
 *
 * Arguments, results, routes, flags and errors are those of aps_sync.  In
 * addition, a set whose aps_sync_workspace_bytes(n, L) exceeds
 * APS_SYNC_SCRATCH_BYTES returns APS_ERR_SIZE before anything is enqueued
 * (96 MiB holds sets up to about 33 M elements, e.g. the 25.6 M of a
 * ResNet-50).  The stream must belong to the current device.
 *
 * Every call on one GPU uses that GPU's one array, whose contents the call
 * does not rely on (each pass writes what it later reads).  Calls that
 * overlap on one GPU (two streams, two threads, or pass 1 of one set issued
 * between pass 1 and pass 2 of another) race on it and give undefined
 * results; serialise them.
 */
#define APS_SYNC_SCRATCH_BYTES ((uint64_t)96 << 20)
int aps_sync_noalloc(const float* G, int32_t W, int64_t ld, int64_t n,
                     const int64_t* offsets, int32_t L,
                     const aps_format* fmts, int32_t n_fmts, const uint8_t* fmt_idx,
                     uint32_t flags, uint32_t* maxabs_bits, int32_t* scale_exp, float* out,
                     void* stream);

/* Summation order and accumulator of aps_sim_reduce_ex. */
enum { APS_ACC_SEQUENTIAL = 0, APS_ACC_KAHAN = 1 };
typedef struct {
    int32_t group;       /* group size k of the hierarchical all-reduce: a power of
                            two dividing W.  k = W: one group, worker order 0..W-1;
                            k = 1: a ring all-reduce over all W workers */
    int32_t accumulator; /* APS_ACC_SEQUENTIAL: s = R(s + x); APS_ACC_KAHAN:
                            Kahan's compensated summation, every operation
                            rounded to the format */
} aps_reduce_opts;

/*
 * aps_sim_reduce with the summation order of the hierarchical all-reduce of
 * Sec. 4.2 and an accumulation strategy of CPD (Sec. 5):
 *   - the W workers form W/k groups of k consecutive workers; each group's
 *     master (its first worker) sums the group in worker order;
 *   - the masters then run a ring all-reduce on the group sums: element j
 *     lies in ring segment s = floor(j * (W/k) / n), and segment s adds the
 *     group sums in master order s, s+1, ..., s + W/k - 1 (mod W/k);
 *   - every add of both chains is rounded to the format (or is one step of
 *     Kahan's compensated summation with every operation rounded).
 * opts == NULL is {k = W, APS_ACC_SEQUENTIAL}, i.e. aps_sim_reduce.
 * A k that is not a power of two dividing W returns APS_ERR_SIZE; an unknown
 * accumulator APS_ERR_UNSUPPORTED.  Other arguments as for aps_sim_reduce.
 */
int aps_sim_reduce_ex(const float* G, int32_t W, int64_t ld, int64_t n,
                      const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                      const aps_format* fmts, int32_t n_fmts, const uint8_t* fmt_idx,
                      uint32_t flags, const aps_reduce_opts* opts, float* out, void* codes_out,
                      void* stream);

/*
 * The SUM all-reduce of Algorithm 1 on the cast gradients in the form the
 * workers would exchange them: W rows of packed codes of already scaled and
 * cast values (as written by aps_quantize), summed in worker order with the
 * accumulator rounded to the format after every add (Sec. 5), then cast back
 * and unscaled:
 *   s = decode(c_0[j]);  s = R_fmt(s + decode(c_w[j])) for w = 1..W-1
 *   out[j] = fl32(s / 2^ft)            (s itself with APS_OUTPUT_SCALED)
 * It is the kernel each owner of a slice would run in a multi-GPU
 * reduce-scatter of codes; for 5..8-bit formats it reads one byte per
 * element-worker instead of four.
 *
 *   codes      W rows of packed codes, 16-byte aligned; the row stride is the
 *              code bytes of ld elements (ld/2, ld or 2*ld), which must be a
 *              multiple of 16 bytes
 *   flags      0 or APS_OUTPUT_SCALED
 *   out        fp32[n] out (16-byte aligned), or NULL
 *   codes_out  packed codes of the scaled sum s, [n] (16-byte aligned), or NULL
 */
int aps_sim_reduce_codes(const void* codes, int32_t W, int64_t ld, int64_t n,
                         const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                         const aps_format* fmts, int32_t n_fmts, const uint8_t* fmt_idx,
                         uint32_t flags, float* out, void* codes_out, void* stream);

/*
 * Back to fp32 with the scale undone (Algorithm 1's last two steps):
 *   out[j] = fl32(V[j] / 2^scale_exp[i])
 * where V is Q (fp32 values) if Q is non-NULL, else the decoded codes.
 *
 *   Q          fp32[n] (16-byte aligned) or NULL
 *   codes      packed codes [n] (16-byte aligned), used when Q is NULL
 *   out        fp32[n] out (16-byte aligned), may be Q itself
 */
int aps_dequantize(const float* Q, const void* codes, int64_t n,
                   const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                   const aps_format* fmts, int32_t n_fmts, const uint8_t* fmt_idx,
                   float* out, void* stream);

/*
 * A matrix product on a multiply-accumulate unit of a chosen low precision,
 * CPD's low-precision-accumulator GEMM (Sec. 5): C = A * B with
 *   a = R_in(A[i][k]), b = R_in(B[k][j])       (inputs cast to in_fmt)
 *   p_k = R_acc(a * b)                          (each product cast to acc_fmt)
 *   s = p_0;  s = R_acc(s + p_k) for k = 1..K-1 (sequential, k order), or
 *   Kahan's compensated summation with every operation rounded to acc_fmt
 *   C[i][j] = s                                 (K = 0 gives +0)
 * R_* round to nearest even as described above (overflow to INF, gradual
 * underflow).  Row-major device arrays: A[M][lda], B[K][ldb], C[M][ldc];
 * C must not overlap A or B.
 *
 *   accumulator  APS_ACC_SEQUENTIAL or APS_ACC_KAHAN
 *
 * The product of two in_fmt values is formed exactly in fp32 and then
 * rounded, which needs in_fmt.m <= 11, and either every product of two
 * in_fmt values a multiple of 2^-149 (2 * (emin_in - m_in) >= -149) or
 * every product too small for that rounding to zero in acc_fmt
 * (2 * (m_in + 1) <= emin_acc - m_acc + 149); other pairs, and formats
 * rounded in fp64 (see aps_format_supported), return APS_ERR_UNSUPPORTED.
 * M, N, K in [0, 2^22]; lda >= K, ldb >= N,
 * ldc >= N; A and B may be NULL when K = 0 or M * N = 0.
 * When acc_fmt is IEEE half (e = 5, m = 10, bias 15) and every in_fmt value
 * is a half, the products and adds run on the GPU's half-precision
 * arithmetic, which rounds exactly as above: the results are the same.
 * Likewise in_fmt 1-5-2 (bias 15) and 1-4-3 (bias 7) are cast by the GPU's
 * conversions to the 8-bit floats E5M2 and E4M3 and back (for 1-4-3 with
 * INF from 248 up), which give this cast on every fp32 input.
 */
#define APS_MAX_GEMM_DIM (1 << 22)
int aps_lp_gemm(const float* A, int64_t lda, const float* B, int64_t ldb, float* C, int64_t ldc,
                int32_t M, int32_t N, int32_t K, aps_format in_fmt, aps_format acc_fmt,
                int32_t accumulator, void* stream);

/* Static text for a status code. */
const char* aps_strerror(int status);

#ifdef __cplusplus
}
#endif
#endif /* APS_H */
