/*
 * oracle.c -- CPU oracle for the Auto-Precision-Scaling (APS) gradient path.
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke
 * check and the CPU-baseline leg of the benchmark may load this library.
 * It shares no code with the HIP library and nothing in the product calls it.
 *
 * Plain, slow, scalar C99.  All rounding is done on exact real values held in
 * double precision with frexp / ldexp / nearbyint (default rounding mode, i.e.
 * round-half-to-even).  The only parallelism is an OpenMP loop over
 * independent elements; the arithmetic per element is the paper's, in the
 * paper's order.
 *
 * Paper: Han, Demmel, You, "Auto-Precision Scaling for Distributed Deep
 * Learning", arXiv 1911.08907.  Cited below by section, algorithm, equation
 * and table.
 *
 * Readings of the paper used here (the paper is silent or loose on these):
 *  R1 Format layout (Algorithm 1 names only exp_bit and man_bit): IEEE-754
 *     style -- bias 2^(e-1)-1 by default, gradual underflow (subnormals), the
 *     all-ones exponent reserved for INF/NaN.  With it the five rows of
 *     Table 2 come out exactly.
 *  R2 Overflow (Sec. 3.2 says values above 2^15 overflow for (5,2)): IEEE
 *     round-to-nearest overflow -- a value becomes INF when rounding it with
 *     an unbounded exponent gives a magnitude above the largest finite value.
 *  R3 Underflow (Sec. 3.2 says values below 2^-16 become 0 for (5,2)):
 *     round-to-nearest-even onto the subnormal grid, so only magnitudes up to
 *     half the smallest subnormal become (signed) zero.
 *  R4 Ties when m = 0: "even" is taken as an even multiple of the quantum,
 *     so a significand 1.1b rounds up to 10b.
 *  R5 Signed zeros and NaN follow IEEE-754 arithmetic.
 *  R6 All-zero (or empty) layers and layers whose max magnitude is INF/NaN,
 *     or whose fl32(N * max) overflows, get the scale exponent 0.
 *  R7 The SUM all-reduce runs in worker order 0..W-1 and rounds its
 *     accumulator to the same format after every add (Sec. 5, CPD's
 *     low-precision accumulator); the result is the sum, not the mean.
 *  R8 The scale exponent uses emax = 2^e - 2 - bias, which is Algorithm 1's
 *     upper_bound_exp when the bias is the default.
 */
#include "oracle.h"

#include <limits.h>
#include <math.h>
#include <string.h>

static float f_of_bits(uint32_t b) {
    float f;
    memcpy(&f, &b, sizeof f);
    return f;
}

static uint32_t bits_of_f(float f) {
    uint32_t b;
    memcpy(&b, &f, sizeof b);
    return b;
}

/* ---------------------------------------------------------------- format */

int oracle_emin(oracle_format f) { return 1 - f.bias; }

int oracle_emax(oracle_format f) { return (1 << f.e) - 2 - f.bias; }

/* largest finite value (2 - 2^-m) * 2^emax */
double oracle_maxfinite(oracle_format f) {
    return ldexp(2.0 - ldexp(1.0, -f.m), oracle_emax(f));
}

/* smallest positive (subnormal) value 2^(emin - m); Table 2's lower range end */
double oracle_minsub(oracle_format f) { return ldexp(1.0, oracle_emin(f) - f.m); }

int oracle_format_ok(oracle_format f) {
    if (f.e < 2 || f.e > 8 || f.m < 0 || f.m > 23) return 0;
    if (oracle_emax(f) > 127) return 0;
    if (oracle_emin(f) > oracle_emax(f)) return 0;
    if (oracle_emin(f) - f.m < -149) return 0;
    return 1;
}

/* ------------------------------------------------------------- rounding */

/* The cast to the custom format that Algorithm 1 applies to the scaled
 * gradient, with the round-to-nearest-even mode of Sec. 4 and readings
 * R1-R5.  y is any real held exactly in a double.
 *
 * For a = |y| in the binade [2^E, 2^(E+1)) the format spaces its values by
 * the quantum 2^(max(E, emin) - m); the result is the multiple of that
 * quantum nearest to a (ties to the even multiple), or INF when that
 * multiple exceeds the largest finite value. */
double oracle_round(double y, oracle_format f) {
    if (isnan(y) || isinf(y) || y == 0.0) return y;
    const int emin = oracle_emin(f);
    const double a = fabs(y);
    int E;
    (void)frexp(a, &E); /* a = r * 2^E with r in [0.5, 1) */
    E -= 1;             /* so that a is in [2^E, 2^(E+1)) */
    const int Eq = E > emin ? E : emin;
    const double k = nearbyint(ldexp(a, f.m - Eq)); /* a / quantum, exact scaling */
    double v = ldexp(k, Eq - f.m);
    if (v > oracle_maxfinite(f)) v = INFINITY;
    return copysign(v, y); /* an underflow to zero keeps the sign of y (R5) */
}

/* --------------------------------------------------------------- scales */

int oracle_ceil_log2(double t) {
    int E;
    const double r = frexp(t, &E); /* t = r * 2^E, r in [0.5, 1) */
    return (r == 0.5) ? E - 1 : E; /* exact power of two: log2 t = E - 1 */
}

/* The exponent of one element of the tensor that Algorithm 1 hands to its
 * exponent search, the gradient multiplied by the worker count: the fp32
 * product v = fl32(N * g) has exponent ceil(log2 |v|) (Sec. 3.3.3).  A zero
 * has none (INT32_MIN); an INF or NaN product sets *nonfinite. */
static int32_t product_exponent(float g, int32_t N, int32_t* nonfinite) {
    const float v = (float)N * g;
    if (!isfinite(v)) {
        *nonfinite = 1;
        return INT32_MIN;
    }
    return v == 0.0f ? INT32_MIN : oracle_ceil_log2(fabs((double)v));
}

/* Sec. 3.3.3's exponent of a tensor taken element by element: the largest
 * product_exponent over the tensor.  It is the route Algorithm 1 describes,
 * kept beside the max-abs route (oracle_layer_maxabs, oracle_scale_one) so
 * that a test can show the two agree. */
int32_t oracle_find_max_exp(const float* g, int64_t cnt, int32_t N, int32_t* nonfinite) {
    int32_t e = INT32_MIN;
    *nonfinite = 0;
    for (int64_t k = 0; k < cnt; ++k) {
        const int32_t ek = product_exponent(g[k], N, nonfinite);
        e = ek > e ? ek : e;
    }
    return e;
}

void oracle_layer_maxabs(const float* G, int32_t W, int64_t ld, int64_t n,
                         const int64_t* offsets, int32_t L, uint32_t* maxabs_bits) {
    (void)n;
    for (int32_t i = 0; i < L; ++i) {
        double best = 0.0;
        int saw_nan = 0;
        for (int32_t w = 0; w < W; ++w) {
            const float* row = G + (int64_t)w * ld;
            for (int64_t j = offsets[i]; j < offsets[i + 1]; ++j) {
                const float x = row[j];
                if (isnan(x))
                    saw_nan = 1;
                else if (fabs((double)x) > best)
                    best = fabs((double)x);
            }
        }
        maxabs_bits[i] = saw_nan ? 0x7FC00000u : bits_of_f((float)best);
    }
}

/* Sec. 3.3.3: the scale factor is f = 2^ft with
 *     ft = log2(p) - ceil(log2 |N * ghat|),   p = 2^emax.
 * Algorithm 1 takes the largest exponent of N * g per worker, the MAX over
 * workers, and subtracts it from the format's largest exponent; taking the
 * MAX over workers and elements on ghat first gives the same number, since
 * both fl32(N*x) and ceil(log2 .) are monotone in |x|. */
int32_t oracle_scale_one(uint32_t maxabs_bits, int32_t N, oracle_format f) {
    const float ghat = f_of_bits(maxabs_bits & 0x7FFFFFFFu);
    if (!(ghat > 0.0f) || !isfinite(ghat)) return 0;            /* R6 */
    const float t = (float)((double)N * (double)ghat);            /* fl32(N * ghat) */
    if (!isfinite(t)) return 0;                                   /* R6 */
    return oracle_emax(f) - oracle_ceil_log2((double)t);
}

void oracle_layer_scales(const uint32_t* maxabs_bits, int32_t L, int32_t N,
                         const oracle_format* fmts, const uint8_t* fmt_idx,
                         int32_t* scale_exp) {
    for (int32_t i = 0; i < L; ++i) {
        const oracle_format f = fmts[fmt_idx ? fmt_idx[i] : 0];
        scale_exp[i] = oracle_scale_one(maxabs_bits[i], N, f);
    }
}

/* ------------------------------------------------------- quantize/reduce */

/* Algorithm 1 multiplies the fp32 gradient by 2^ft; the product is the fp32
 * value nearest to x * 2^ft (a single rounding, exact unless the result
 * leaves fp32's normal range). */
static float scale_fp32(float x, int32_t ft) { return (float)ldexp((double)x, ft); }

void oracle_quantize(const float* X, int32_t W, int64_t ld, int64_t n,
                     const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                     const oracle_format* fmts, const uint8_t* fmt_idx, float* Q) {
    (void)n;
    for (int32_t i = 0; i < L; ++i) {
        const oracle_format f = fmts[fmt_idx ? fmt_idx[i] : 0];
        const int32_t ft = scale_exp ? scale_exp[i] : 0;
        for (int32_t w = 0; w < W; ++w) {
            const int64_t base = (int64_t)w * ld;
#pragma omp parallel for schedule(static)
            for (int64_t j = offsets[i]; j < offsets[i + 1]; ++j)
                Q[base + j] = (float)oracle_round((double)scale_fp32(X[base + j], ft), f);
        }
    }
}

void oracle_sim_reduce(const float* G, int32_t W, int64_t ld, int64_t n,
                       const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                       const oracle_format* fmts, const uint8_t* fmt_idx,
                       uint32_t flags, float* out) {
    (void)n;
    for (int32_t i = 0; i < L; ++i) {
        const oracle_format f = fmts[fmt_idx ? fmt_idx[i] : 0];
        const int32_t ft = scale_exp ? scale_exp[i] : 0;
#pragma omp parallel for schedule(static)
        for (int64_t j = offsets[i]; j < offsets[i + 1]; ++j) {
            double s = 0.0;
            for (int32_t w = 0; w < W; ++w) {
                const float x = G[(int64_t)w * ld + j];
                /* the scale by 2^ft (not when the input is already scaled) */
                const float y = (flags & ORACLE_INPUT_QUANTIZED) ? x : scale_fp32(x, ft);
                /* the cast to the format */
                const double q = oracle_round((double)y, f);
                /* the SUM all-reduce in worker order with a low-precision
                 * accumulator (Sec. 5): every partial sum is rounded to the
                 * format.  The double add of two format values followed by
                 * one rounding equals rounding the exact sum (53 >= 2*24 + 2). */
                s = (w == 0) ? q : oracle_round(s + q, f);
            }
            /* back to fp32: s is a format value, hence exactly an fp32 value */
            const float g = (float)s;
            /* the scale undone */
            out[j] = (flags & ORACLE_OUTPUT_SCALED) ? g : (float)ldexp((double)g, -ft);
        }
    }
}

/* ----------------------------------------------------------------- codes */

uint32_t oracle_encode(double v, oracle_format f) {
    const uint32_t sign = signbit(v) ? 1u : 0u;
    const uint32_t expmax = (1u << f.e) - 1u;
    uint32_t ef, mant;
    if (isnan(v)) {
        ef = expmax;
        mant = f.m > 0 ? (1u << (f.m - 1)) : 0u; /* quiet NaN; no NaN code when m = 0 */
    } else if (isinf(v)) {
        ef = expmax;
        mant = 0u;
    } else {
        const double a = fabs(v);
        const int emin = oracle_emin(f);
        if (a < ldexp(1.0, emin)) { /* subnormal or zero: a = mant * 2^(emin-m) */
            ef = 0u;
            mant = (uint32_t)ldexp(a, f.m - emin);
        } else { /* a = (1 + mant/2^m) * 2^E */
            int E;
            (void)frexp(a, &E);
            E -= 1;
            ef = (uint32_t)(E + f.bias);
            mant = (uint32_t)ldexp(ldexp(a, -E) - 1.0, f.m);
        }
    }
    return (sign << (f.e + f.m)) | (ef << f.m) | mant;
}

double oracle_decode(uint32_t code, oracle_format f) {
    const uint32_t expmax = (1u << f.e) - 1u;
    const uint32_t sign = (code >> (f.e + f.m)) & 1u;
    const uint32_t ef = (code >> f.m) & expmax;
    const uint32_t mant = code & ((1u << f.m) - 1u);
    double a;
    if (ef == expmax)
        a = mant == 0u ? INFINITY : NAN;
    else if (ef == 0u)
        a = ldexp((double)mant, oracle_emin(f) - f.m);
    else
        a = ldexp(1.0 + ldexp((double)mant, -f.m), (int)ef - f.bias);
    return sign ? -a : a;
}

static int code_bits(oracle_format f) { return 1 + f.e + f.m; }

static void put_code(void* codes, int64_t j, uint32_t c, int bits) {
    uint8_t* b = (uint8_t*)codes;
    if (bits <= 4) {
        const int shift = (int)(j & 1) * 4;
        b[j >> 1] = (uint8_t)((b[j >> 1] & ~(0xF << shift)) | ((c & 0xF) << shift));
    } else if (bits <= 8) {
        b[j] = (uint8_t)c;
    } else {
        b[2 * j] = (uint8_t)(c & 0xFF);
        b[2 * j + 1] = (uint8_t)(c >> 8);
    }
}

static uint32_t get_code(const void* codes, int64_t j, int bits) {
    const uint8_t* b = (const uint8_t*)codes;
    if (bits <= 4) return (b[j >> 1] >> ((int)(j & 1) * 4)) & 0xFu;
    if (bits <= 8) return b[j];
    return (uint32_t)b[2 * j] | ((uint32_t)b[2 * j + 1] << 8);
}

void oracle_pack_codes(const float* V, int64_t n, const int64_t* offsets, int32_t L,
                       const oracle_format* fmts, const uint8_t* fmt_idx, void* codes) {
    (void)n;
    for (int32_t i = 0; i < L; ++i) {
        const oracle_format f = fmts[fmt_idx ? fmt_idx[i] : 0];
        for (int64_t j = offsets[i]; j < offsets[i + 1]; ++j)
            put_code(codes, j, oracle_encode((double)V[j], f), code_bits(f));
    }
}

void oracle_dequantize(const float* Q, const void* codes, int64_t n,
                       const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                       const oracle_format* fmts, const uint8_t* fmt_idx, float* out) {
    (void)n;
    for (int32_t i = 0; i < L; ++i) {
        const oracle_format f = fmts[fmt_idx ? fmt_idx[i] : 0];
        const int32_t ft = scale_exp ? scale_exp[i] : 0;
        for (int64_t j = offsets[i]; j < offsets[i + 1]; ++j) {
            const double v = Q ? (double)Q[j] : oracle_decode(get_code(codes, j, code_bits(f)), f);
            out[j] = (float)ldexp(v, -ft); /* back to fp32, the scale undone */
        }
    }
}

/* byte offset of element j's code in a row, and the row stride in bytes */
static int64_t code_row_bytes(int64_t ld, int bits) {
    return bits <= 4 ? ld / 2 : (bits <= 8 ? ld : 2 * ld);
}

void oracle_sim_reduce_codes(const void* codes, int32_t W, int64_t ld, int64_t n,
                             const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                             const oracle_format* fmts, const uint8_t* fmt_idx,
                             uint32_t flags, float* out) {
    (void)n;
    const uint8_t* base = (const uint8_t*)codes;
    for (int32_t i = 0; i < L; ++i) {
        const oracle_format f = fmts[fmt_idx ? fmt_idx[i] : 0];
        const int bits = code_bits(f);
        const int64_t stride = code_row_bytes(ld, bits);
        const int32_t ft = scale_exp ? scale_exp[i] : 0;
#pragma omp parallel for schedule(static)
        for (int64_t j = offsets[i]; j < offsets[i + 1]; ++j) {
            double s = 0.0;
            for (int32_t w = 0; w < W; ++w) {
                const double q = oracle_decode(get_code(base + w * stride, j, bits), f);
                s = (w == 0) ? q : oracle_round(s + q, f); /* low-precision accumulator */
            }
            const float g = (float)s;
            out[j] = (flags & ORACLE_OUTPUT_SCALED) ? g : (float)ldexp((double)g, -ft);
        }
    }
}

/* ---------------------------------------------- summation order, Kahan */

/* One add of a chain: plain (s = R(s + x)) or Kahan, where every
 * intermediate is cast to the format as a low-precision accumulator would
 * hold it (Sec. 5). */
static void chain_add(double* s, double* c, double x, oracle_format f, int32_t accumulator) {
    if (accumulator == ORACLE_ACC_KAHAN) {
        const double y = oracle_round(x - *c, f);
        const double t = oracle_round(*s + y, f);
        *c = oracle_round(oracle_round(t - *s, f) - y, f);
        *s = t;
    } else {
        *s = oracle_round(*s + x, f);
    }
}

void oracle_sim_reduce_ex(const float* G, int32_t W, int64_t ld, int64_t n,
                          const int64_t* offsets, int32_t L, const int32_t* scale_exp,
                          const oracle_format* fmts, const uint8_t* fmt_idx,
                          uint32_t flags, int32_t group, int32_t accumulator, float* out) {
    const int32_t k = group;
    const int32_t ng = W / k; /* number of groups (masters) */
    for (int32_t i = 0; i < L; ++i) {
        const oracle_format f = fmts[fmt_idx ? fmt_idx[i] : 0];
        const int32_t ft = scale_exp ? scale_exp[i] : 0;
#pragma omp parallel for schedule(static)
        for (int64_t j = offsets[i]; j < offsets[i + 1]; ++j) {
            const int64_t seg = j * ng / n; /* ring segment of this element */
            double T = 0.0, cT = 0.0;
            for (int32_t gi = 0; gi < ng; ++gi) {
                const int32_t g = (int32_t)((seg + gi) % ng);
                double S = 0.0, cS = 0.0;
                for (int32_t m = 0; m < k; ++m) {
                    const float x = G[(int64_t)(g * k + m) * ld + j];
                    const float y = (flags & ORACLE_INPUT_QUANTIZED) ? x : scale_fp32(x, ft);
                    const double q = oracle_round((double)y, f);
                    if (m == 0)
                        S = q; /* the master's own gradient */
                    else
                        chain_add(&S, &cS, q, f, accumulator);
                }
                if (gi == 0)
                    T = S; /* the ring starts at master seg */
                else
                    chain_add(&T, &cT, S, f, accumulator);
            }
            const float gv = (float)T;
            out[j] = (flags & ORACLE_OUTPUT_SCALED) ? gv : (float)ldexp((double)gv, -ft);
        }
    }
}

/* ------------------------------------ low-precision-accumulator GEMM */

/* Sec. 5 (CPD): a matrix product whose multiply-accumulate unit works in a
 * low-precision format.  Each input element is cast to `in` (x -> Cast_in(x)),
 * each product of two cast inputs is cast to the accumulator format `acc`,
 * and the products of one output are accumulated in k order 0..K-1 by a
 * chain of adds in `acc` (plain or Kahan, every intermediate cast).  The
 * product of two values of at most 24 significant bits is exact in double,
 * so each cast below rounds an exact real value once.  K = 0 gives +0. */
void oracle_lp_gemm(const float* A, int64_t lda, const float* B, int64_t ldb, float* C, int64_t ldc,
                    int32_t M, int32_t N, int32_t K, oracle_format in, oracle_format acc,
                    int32_t accumulator) {
#pragma omp parallel for schedule(static)
    for (int32_t i = 0; i < M; ++i) {
        for (int32_t j = 0; j < N; ++j) {
            double s = 0.0, c = 0.0;
            for (int32_t k = 0; k < K; ++k) {
                const double a = oracle_round((double)A[(int64_t)i * lda + k], in);
                const double b = oracle_round((double)B[(int64_t)k * ldb + j], in);
                const double p = oracle_round(a * b, acc); /* the product, held in acc */
                if (k == 0)
                    s = p;
                else
                    chain_add(&s, &c, p, acc, accumulator);
            }
            C[(int64_t)i * ldc + j] = (float)s;
        }
    }
}

double oracle_round_off_error(const float* grad_h, const float* grad_l, int64_t n) {
    double sum = 0.0;
    int64_t cnt = 0;
    for (int64_t j = 0; j < n; ++j) {
        if (grad_h[j] == 0.0f) continue;
        sum += fabs(((double)grad_h[j] - (double)grad_l[j]) / (double)grad_h[j]);
        ++cnt;
    }
    return cnt ? sum / (double)cnt : 0.0;
}
