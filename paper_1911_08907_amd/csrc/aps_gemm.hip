// aps_gemm.hip -- a GEMM on a multiply-accumulate unit of a chosen low
// precision, CPD's low-precision-accumulator GEMM (Sec. 5).
#include "aps_common.hpp"

namespace aps {

// ================================================== K6: low-precision GEMM

struct GemmArgs {
    const float* __restrict__ A;
    const float* __restrict__ B;
    float* __restrict__ C;
    int64_t lda, ldb, ldc;
    int32_t M, N, K;
    int32_t ka, kb;  // staged A and B carry 2^ka, 2^kb (ka + kb = k of the accumulator, or both 0)
    int64_t tiles;   // output tiles, ntn of them per row of tiles (n fastest)
    int32_t ntn;
    float qs;        // GP_GRID: 2^Q, the accumulator's subnormal step in its working domain
};

// How a product reaches the accumulator's working domain and is rounded:
enum GemmProduct {
    GP_LDEXP = 0,   // operands native: fl32(a * b) then 2^k, rounded (quant)
    GP_SCALED = 1,  // operands pre-scaled at staging: a_w * b_w rounded (quant_w)
    GP_FIT = 2,     // pre-scaled, and every product fits the significand (quant_fit)
    GP_GRID = 3,    // as GP_FIT, staged so that the subnormal step is 1: rint, then 2^Q
    GP_EXACT = 4,   // pre-scaled, every product fits and none reaches the subnormal range: no rounding
    GP_BF16 = 5,    // GP_EXACT into bfloat16: each add rounded by the hardware's conversion to bfloat16
};

// GP_BF16.  The accumulator is bfloat16 (e = 8, m = 7, bias 127): its values
// are the fp32 values whose low 16 bits are zero, and fp32's own
// round-to-nearest-even conversion to bfloat16 (subnormals and overflow to
// INF included) is the format's rounding.  The fp32 add of two bfloat16
// values rounded once more to bfloat16 is the rounded exact sum (24 >=
// 2 * 8 + 2), so each add is an fp32 add and a conversion, one packed
// conversion for two chains.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void round_bf16x2(float x0, float x1, float& r0, float& r1) {
    const uint32_t u = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{x0, x1}, bf16x2));
    r0 = u2f(u << 16);
    r1 = u2f(u & 0xFFFF0000u);
}

// GP_EXACT.  When every product of two input values fits the accumulator's
// significand and no nonzero product lies below 2^emin (the square of the
// input's smallest subnormal is at least 2^emin), every product is already
// a format value, or beyond the largest one, where the working domain makes
// it INF as fp32 does: the exact fp32 product is its own rounding.

// GP_GRID.  A product of two input values that fits the accumulator's
// significand is, from 2^emin up, already a multiple of the accumulator's
// subnormal step 2^(emin - m); below 2^emin the format rounds it to the
// nearest such multiple, ties to even.  So on a scale where that step is 1
// its rounding is one round-to-nearest-even to an integer at every
// magnitude, with no compare and select between the normal and subnormal
// cases.  The operands are staged with 2^(m - emin) between them, the
// product is rounded by rint, and 2^Q (Q = the step's exponent in the
// working domain, >= 0) carries it into the working domain: exactly, or to
// INF where the product overflows the format, as the format's own
// overflow threshold sits at fp32's there.  A staged product below 2^-126
// is below 1/2 and rounds to a signed zero whatever fp32 made of it.

constexpr int GT = 64;  // output tile GT x GT per block, 4 x 4 per thread
constexpr int GK = 16;  // k-tile staged in LDS

// Input format 1-5-2 with bias 15 has the bit layout and value set of the
// OCP E5M2 8-bit float.  The hardware's conversion of fp32 to it (round to
// nearest even, no saturation: beyond the largest finite value the result is
// INF, a NaN stays NaN, subnormals kept) and back to fp32 is this format's
// cast exactly; the two agree on every fp32 bit pattern.  Two values per
// conversion.
constexpr int VI_E5M2 = 100;

__device__ __forceinline__ void cast_e5m2x2(float x0, float x1, float& r0, float& r1) {
    const int pk = __builtin_amdgcn_cvt_pk_bf8_f32(x0, x1, 0, false);  // bytes 0 and 1
    const f32x2 v = __builtin_amdgcn_cvt_pk_f32_bf8(pk, false);
    r0 = v[0];
    r1 = v[1];
}

// Input format 1-4-3 with bias 7 shares its layout, subnormals and rounding
// with the OCP E4M3 8-bit float below 248; E4M3 has no INF and goes on to
// 448, so from 248 up (the tie at 248 rounds to 256) the cast is INF with the
// input's sign, which also covers an INF input.  With that one select the
// round trip is this format's cast on every fp32 bit pattern.
constexpr int VI_E4M3 = 101;

__device__ __forceinline__ void cast_e4m3x2(float x0, float x1, float& r0, float& r1) {
    const int pk = __builtin_amdgcn_cvt_pk_fp8_f32(x0, x1, 0, false);  // bytes 0 and 1
    const f32x2 v = __builtin_amdgcn_cvt_pk_f32_fp8(pk, false);
    r0 = __builtin_fabsf(x0) >= 248.0f ? __builtin_copysignf(__builtin_inff(), x0) : v[0];
    r1 = __builtin_fabsf(x1) >= 248.0f ? __builtin_copysignf(__builtin_inff(), x1) : v[1];
}

// Two input values cast by the hardware conversion of the launch's mode.
template <int VI>
__device__ __forceinline__ void cast_hw_x2(float x0, float x1, float& r0, float& r1) {
    if constexpr (VI == VI_E5M2)
        cast_e5m2x2(x0, x1, r0, r1);
    else
        cast_e4m3x2(x0, x1, r0, r1);
}

// The launch's input mode: a hardware conversion, or the format's class.
inline bool input_mode_is(int vi, const FmtK& f) {
    if (vi == VI_E5M2) return f.e == 5 && f.m == 2 && f.bias == 15;
    if (vi == VI_E4M3) return f.e == 4 && f.m == 3 && f.bias == 7;
    return f.variant == vi;
}

// An input value cast to the input format (native value): through the
// switch over classes, straight to the class VI when the launch knows it, or
// by a hardware conversion (E5M2, E4M3).
template <int VI>
__device__ __forceinline__ float cast_in(float x, const FmtK& fi) {
    if constexpr (VI == VI_E5M2 || VI == VI_E4M3) {
        float r, unused;
        cast_hw_x2<VI>(x, x, r, unused);
        return r;
    } else if constexpr (VI < 0) {
        return quant_any(x, fi.k, fi);
    } else {
        return quant_native<VI>(x, fi.k, fi);
    }
}

// One block computes a GT x GT tile of C.  Each k-tile of A and B is cast to
// the input format while it is staged into LDS (A transposed, so a thread's
// four rows are one 16-byte read); each thread then runs 16 independent
// chains, one per output, adding its products in k order.  The work is the
// VALU's: a product, its rounding and the rounded add per multiply-accumulate.
template <int V, bool KAHAN, int PM, int VI = -1>
__global__ __launch_bounds__(BLOCK) void k_lp_gemm(GemmArgs g, FmtK fi, FmtK fa) {
    __shared__ __align__(16) float As[GK][GT + 4];  // As[k][m]; the pad spreads the staging writes over banks
    __shared__ __align__(16) float Bs[GK][GT + 4];  // Bs[k][n]
    const int t = threadIdx.x;
    const int tx = t & 15, ty = t >> 4;
    // a 1-D grid over the tiles (a grid's y extent is limited to 65535 blocks);
    // a block takes a further tile only where the tiles outnumber the grid
    for (int64_t tile = blockIdx.x; tile < g.tiles; tile += gridDim.x) {
        const int64_t m0 = tile / g.ntn * GT, n0 = tile % g.ntn * GT;
        float s[4][4], c[4][4];
        bool bad[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                s[i][j] = 0.0f;
                c[i][j] = 0.0f;
                bad[i][j] = false;
            }
        float ra[4], rb[4];
        // Staged value r of this thread: A[m0 + t/16 + 16r][k0 + t%16] and B[k0 + t/64 + 4r][n0 + t%64].
        const bool inner = m0 + GT <= g.M && n0 + GT <= g.N;  // the tile lies inside C
        const int64_t oa = (m0 + (t >> 4)) * g.lda + (t & 15);  // offsets of value 0 in A and B
        const int64_t ob = (int64_t)(t >> 6) * g.ldb + n0 + (t & 63);
        // global -> registers, cast to the input format; outside A and B: 0
        auto fetch = [&](int64_t k0) {
            if (inner && k0 + GK <= g.K) {  // the whole k-tile inside A and B: no checks
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    ra[r] = __builtin_amdgcn_ldexpf(cast_in<VI>(g.A[oa + r * 16 * g.lda + k0], fi), g.ka);
                    rb[r] = __builtin_amdgcn_ldexpf(cast_in<VI>(g.B[ob + (k0 + 4 * r) * g.ldb], fi), g.kb);
                }
                return;
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int idx = t + BLOCK * r;
                const int64_t am = m0 + (idx >> 4), ak = k0 + (idx & 15);
                ra[r] = (am < g.M && ak < g.K) ? __builtin_amdgcn_ldexpf(cast_in<VI>(g.A[am * g.lda + ak], fi), g.ka)
                                               : 0.0f;
                const int64_t bk = k0 + (idx >> 6), bn = n0 + (idx & 63);
                rb[r] = (bk < g.K && bn < g.N) ? __builtin_amdgcn_ldexpf(cast_in<VI>(g.B[bk * g.ldb + bn], fi), g.kb)
                                               : 0.0f;
            }
        };
        auto mac_v = [&](const f4& av, const f4& bv, bool first) {
            const float a[4] = {av.x, av.y, av.z, av.w};
            const float b[4] = {bv.x, bv.y, bv.z, bv.w};
            if constexpr (PM == GP_BF16) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; j += 2) {
                        const float p0 = a[i] * b[j], p1 = a[i] * b[j + 1];  // exact, bfloat16 values or beyond
                        if (first) {
                            s[i][j] = p0;
                            s[i][j + 1] = p1;
                        } else if constexpr (KAHAN) {
                            float y0, y1, t0, t1, u0, u1;
                            round_bf16x2(p0 - c[i][j], p1 - c[i][j + 1], y0, y1);
                            round_bf16x2(s[i][j] + y0, s[i][j + 1] + y1, t0, t1);
                            round_bf16x2(t0 - s[i][j], t1 - s[i][j + 1], u0, u1);
                            round_bf16x2(u0 - y0, u1 - y1, c[i][j], c[i][j + 1]);
                            s[i][j] = t0;
                            s[i][j + 1] = t1;
                        } else {
                            round_bf16x2(s[i][j] + p0, s[i][j + 1] + p1, s[i][j], s[i][j + 1]);
                        }
                    }
                return;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    // exact fp32 product of two input-format values, cast to the accumulator
                    float p;
                    if constexpr (PM == GP_LDEXP)
                        p = quant<V>(a[i] * b[j], fa.k, fa, bad[i][j]);
                    else if constexpr (PM == GP_SCALED)
                        p = quant_w<V>(a[i] * b[j], fa, bad[i][j]);
                    else if constexpr (PM == GP_FIT)
                        p = quant_fit<V>(a[i] * b[j], fa);
                    else if constexpr (PM == GP_GRID)
                        p = __builtin_rintf(a[i] * b[j]) * g.qs;
                    else
                        p = a[i] * b[j];
                    if (first)
                        s[i][j] = p;
                    else
                        chain_step<V, KAHAN>(s[i][j], c[i][j], p, fa, bad[i][j]);
                }
        };
        auto mac = [&](int kk, bool first) {
            mac_v(*(const f4*)&As[kk][ty * 4], *(const f4*)&Bs[kk][tx * 4], first);
        };
        if (g.K > 0) fetch(0);
        for (int64_t k0 = 0; k0 < g.K; k0 += GK) {
            __syncthreads();  // the previous k-tile is consumed
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int idx = t + BLOCK * r;
                As[idx & 15][idx >> 4] = ra[r];
                Bs[idx >> 6][idx & 63] = rb[r];
            }
            __syncthreads();
            if (k0 + GK < g.K) fetch(k0 + GK);  // the next k-tile's loads overlap this tile's math
            const int kend = (int)min((int64_t)GK, g.K - k0);
            if (k0 > 0 && kend == GK) {
                // software-pipelined: step kk+1's LDS reads are issued before step kk's math
                f4 av = *(const f4*)&As[0][ty * 4], bv = *(const f4*)&Bs[0][tx * 4];
#pragma unroll
                for (int kk = 0; kk < GK; ++kk) {
                    f4 an = av, bn = bv;
                    if (kk + 1 < GK) {
                        an = *(const f4*)&As[kk + 1][ty * 4];
                        bn = *(const f4*)&Bs[kk + 1][tx * 4];
                    }
                    __builtin_amdgcn_sched_barrier(0);
                    mac_v(av, bv, false);
                    av = an;
                    bv = bn;
                }
            } else {
                int kk = 0;
                if (k0 == 0) {
                    mac(0, true);  // an output's chain starts with its first product
                    kk = 1;
                }
#pragma unroll 1
                for (; kk < kend; ++kk) mac(kk, false);
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t m = m0 + ty * 4 + i;
            if (m >= g.M) continue;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t n = n0 + tx * 4 + j;
                if (n < g.N) g.C[m * g.ldc + n] = __builtin_amdgcn_ldexpf(finish<V>(s[i][j], bad[i][j]), -fa.k);
            }
        }
    }
}

// ===================================== K6h: the accumulator is IEEE half
//
// When the accumulator is the half-precision format (e = 5, m = 10, bias
// 15) and every input value is a half, the hardware's half-precision
// multiply and add are the emulated unit: each rounds its exact result to
// nearest even, with subnormals and overflow to INF, as the format does.
// So the products and the chain run in packed halves, one multiply and one
// add (Kahan: one multiply, four adds) per two outputs, with no bit
// manipulation.  Nothing may fuse a multiply with the add that follows it.

using h2 = _Float16 __attribute__((ext_vector_type(2)));

constexpr int HT = 4;         // outputs per thread along each side: HT x HT
constexpr int HGT = 16 * HT;  // output tile HGT x HGT per block (16 x 16 threads)
constexpr int HGK = 16;       // k-tile staged in LDS
constexpr int HST = HGT * HGK / BLOCK;  // staged values of A (and of B) per thread and k-tile

template <int N>
struct HVec {
    using T = _Float16 __attribute__((ext_vector_type(N)));
};

template <bool KAHAN, int VI>
__global__ __launch_bounds__(BLOCK) void k_lp_gemm_h(GemmArgs g, FmtK fi) {
#pragma clang fp contract(off)
    using hv = typename HVec<HT>::T;
    __shared__ __align__(16) _Float16 As[HGK][HGT + 8];  // As[k][m]; the pad spreads the staging writes over banks
    __shared__ __align__(16) _Float16 Bs[HGK][HGT + 8];  // Bs[k][n]
    const int t = threadIdx.x;
    const int tx = t & 15, ty = t >> 4;
    for (int64_t tile = blockIdx.x; tile < g.tiles; tile += gridDim.x) {
        const int64_t m0 = tile / g.ntn * HGT, n0 = tile % g.ntn * HGT;
        // output (ty*HT + i, tx*HT + 2*h + e) is element e of s[i][h]
        h2 s[HT][HT / 2], c[HT][HT / 2];
#pragma unroll
        for (int i = 0; i < HT; ++i)
#pragma unroll
            for (int h = 0; h < HT / 2; ++h) {
                s[i][h] = h2{0, 0};
                c[i][h] = h2{0, 0};
            }
        _Float16 ra[HST], rb[HST];
        // Staged value r of this thread: A[m0 + t/HGK + r*BLOCK/HGK][k0 + t%HGK] and
        // B[k0 + t/HGT + r*BLOCK/HGT][n0 + t%HGT].
        const bool inner = m0 + HGT <= g.M && n0 + HGT <= g.N;  // the tile lies inside C
        const int64_t oa = (m0 + t / HGK) * g.lda + t % HGK;  // offsets of value 0 in A and B
        const int64_t ob = (int64_t)(t / HGT) * g.ldb + n0 + t % HGT;
        // global -> registers, cast to the input format (a half, exactly); outside A and B: 0.
        // Every load reads an address inside the matrix, so no lane branches.
        auto fetch = [&](int64_t k0) {
            if (inner && k0 + HGK <= g.K) {  // the whole k-tile inside A and B: no checks
                if constexpr (VI == VI_E5M2 || VI == VI_E4M3) {  // two values per conversion
#pragma unroll
                    for (int r = 0; r < HST; r += 2) {
                        float a0, a1, b0, b1;
                        cast_hw_x2<VI>(g.A[oa + r * (BLOCK / HGK) * g.lda + k0],
                                       g.A[oa + (r + 1) * (BLOCK / HGK) * g.lda + k0], a0, a1);
                        cast_hw_x2<VI>(g.B[ob + (k0 + r * (BLOCK / HGT)) * g.ldb],
                                       g.B[ob + (k0 + (r + 1) * (BLOCK / HGT)) * g.ldb], b0, b1);
                        ra[r] = (_Float16)a0;
                        ra[r + 1] = (_Float16)a1;
                        rb[r] = (_Float16)b0;
                        rb[r + 1] = (_Float16)b1;
                    }
                    return;
                }
#pragma unroll
                for (int r = 0; r < HST; ++r) {
                    ra[r] = (_Float16)cast_in<VI>(g.A[oa + r * (BLOCK / HGK) * g.lda + k0], fi);
                    rb[r] = (_Float16)cast_in<VI>(g.B[ob + (k0 + r * (BLOCK / HGT)) * g.ldb], fi);
                }
                return;
            }
#pragma unroll
            for (int r = 0; r < HST; ++r) {
                const int idx = t + BLOCK * r;
                const int64_t am = m0 + idx / HGK, ak = k0 + idx % HGK;
                const bool oka = am < g.M && ak < g.K;
                const _Float16 qa = (_Float16)cast_in<VI>(g.A[oka ? am * g.lda + ak : 0], fi);
                ra[r] = oka ? qa : (_Float16)0.0f;
                const int64_t bk = k0 + idx / HGT, bn = n0 + idx % HGT;
                const bool okb = bk < g.K && bn < g.N;
                const _Float16 qb = (_Float16)cast_in<VI>(g.B[okb ? bk * g.ldb + bn : 0], fi);
                rb[r] = okb ? qb : (_Float16)0.0f;
            }
        };
        auto step_v = [&](const hv& av, const hv& bv, bool first) {
#pragma unroll
            for (int i = 0; i < HT; ++i) {
                const h2 a = h2{av[i], av[i]};
                h2 p[HT / 2];
#pragma unroll
                for (int h = 0; h < HT / 2; ++h) p[h] = a * h2{bv[2 * h], bv[2 * h + 1]};  // rounded to half
                if (first) {
#pragma unroll
                    for (int h = 0; h < HT / 2; ++h) s[i][h] = p[h];  // a chain starts with its first product
                } else if constexpr (KAHAN) {
                    // each phase over the row's chains in turn, so that no add waits on the one before it
                    h2 y[HT / 2], tt[HT / 2];
#pragma unroll
                    for (int h = 0; h < HT / 2; ++h) y[h] = p[h] - c[i][h];
#pragma unroll
                    for (int h = 0; h < HT / 2; ++h) tt[h] = s[i][h] + y[h];
#pragma unroll
                    for (int h = 0; h < HT / 2; ++h) c[i][h] = tt[h] - s[i][h];
#pragma unroll
                    for (int h = 0; h < HT / 2; ++h) {
                        c[i][h] = c[i][h] - y[h];
                        s[i][h] = tt[h];
                    }
                } else {
#pragma unroll
                    for (int h = 0; h < HT / 2; ++h) s[i][h] = s[i][h] + p[h];
                }
            }
        };
        auto step = [&](int kk, bool first) {
            step_v(*(const hv*)&As[kk][ty * HT], *(const hv*)&Bs[kk][tx * HT], first);
        };
        if (g.K > 0) fetch(0);
        for (int64_t k0 = 0; k0 < g.K; k0 += HGK) {
            __syncthreads();  // the previous k-tile is consumed
#pragma unroll
            for (int r = 0; r < HST; ++r) {
                const int idx = t + BLOCK * r;
                As[idx % HGK][idx / HGK] = ra[r];
                Bs[idx / HGT][idx % HGT] = rb[r];
            }
            __syncthreads();
            if (k0 + HGK < g.K) fetch(k0 + HGK);  // the next k-tile's loads overlap this tile's math
            const int kend = (int)min((int64_t)HGK, g.K - k0);
            if (k0 > 0 && kend == HGK) {
                // software-pipelined: step kk+1's LDS reads are issued before step kk's math
                hv av = *(const hv*)&As[0][ty * HT], bv = *(const hv*)&Bs[0][tx * HT];
#pragma unroll
                for (int kk = 0; kk < HGK; ++kk) {
                    hv an = av, bn = bv;
                    if (kk + 1 < HGK) {
                        an = *(const hv*)&As[kk + 1][ty * HT];
                        bn = *(const hv*)&Bs[kk + 1][tx * HT];
                    }
                    __builtin_amdgcn_sched_barrier(0);
                    step_v(av, bv, false);
                    av = an;
                    bv = bn;
                }
            } else {
                int kk = 0;
                if (k0 == 0) {
                    step(0, true);
                    kk = 1;
                }
#pragma unroll 1
                for (; kk < kend; ++kk) step(kk, false);
            }
        }
#pragma unroll
        for (int i = 0; i < HT; ++i) {
            const int64_t m = m0 + ty * HT + i;
            if (m >= g.M) continue;
#pragma unroll
            for (int j = 0; j < HT; ++j) {
                const int64_t n = n0 + tx * HT + j;
                if (n < g.N) g.C[m * g.ldc + n] = (float)s[i][j >> 1][j & 1];
            }
        }
    }
}

}  // namespace aps

using namespace aps;

template <int V>
static void launch_lp_gemm_v(bool kahan, int pm, dim3 grid, hipStream_t s, const GemmArgs& g, const FmtK& fi,
                             const FmtK& fa) {
    constexpr bool can_fit = (VT<V>::cls == CLS_TOP || VT<V>::cls == CLS_LOW) && !VT<V>::m0;
    constexpr bool can_ldexp = VT<V>::cls == CLS_TOP || VT<V>::cls == CLS_LOW;
    constexpr bool can_exact = VT<V>::cls != CLS_GEN && !VT<V>::m0;
#define APS_G(K, P) hipLaunchKernelGGL((k_lp_gemm<V, K, P>), grid, dim3(BLOCK), 0, s, g, fi, fa)
    if (pm == GP_BF16) {
        if constexpr (V == V_INT_F32) {
            // one instantiation per input class (such inputs are TOP or LOW)
#define APS_GB(VI)                                                                                           \
    if (input_mode_is((VI), fi)) {                                                                                \
        if (kahan)                                                                                           \
            hipLaunchKernelGGL((k_lp_gemm<V, true, GP_BF16, VI>), grid, dim3(BLOCK), 0, s, g, fi, fa);  \
        else                                                                                                 \
            hipLaunchKernelGGL((k_lp_gemm<V, false, GP_BF16, VI>), grid, dim3(BLOCK), 0, s, g, fi, fa); \
        return;                                                                                              \
    }
            APS_GB(VI_E5M2) APS_GB(VI_E4M3) APS_GB(V_TOP_F32) APS_GB(V_TOP_M0) APS_GB(V_LOW_F32) APS_GB(V_LOW_M0)
#undef APS_GB
            if (kahan) APS_G(true, GP_BF16); else APS_G(false, GP_BF16);
            return;
        }
    }
    if (pm == GP_EXACT || pm == GP_BF16) {
        if constexpr (can_exact) {
            if (kahan) APS_G(true, GP_EXACT); else APS_G(false, GP_EXACT);
            return;
        }
    }
    if (pm == GP_GRID) {
        if constexpr (can_fit) {
#define APS_GG(VI)                                                                                           \
    if (input_mode_is((VI), fi)) {                                                                           \
        if (kahan)                                                                                           \
            hipLaunchKernelGGL((k_lp_gemm<V, true, GP_GRID, VI>), grid, dim3(BLOCK), 0, s, g, fi, fa);  \
        else                                                                                                 \
            hipLaunchKernelGGL((k_lp_gemm<V, false, GP_GRID, VI>), grid, dim3(BLOCK), 0, s, g, fi, fa); \
        return;                                                                                              \
    }
            APS_GG(VI_E5M2) APS_GG(VI_E4M3)
#undef APS_GG
            if (kahan) APS_G(true, GP_GRID); else APS_G(false, GP_GRID);
            return;
        }
    }
    if (pm == GP_FIT) {
        if constexpr (can_fit) {
            if (kahan) APS_G(true, GP_FIT); else APS_G(false, GP_FIT);
            return;
        }
    }
    if (pm == GP_LDEXP) {
        if constexpr (can_ldexp) {
            if (kahan) APS_G(true, GP_LDEXP); else APS_G(false, GP_LDEXP);
            return;
        }
    }
    if (kahan) APS_G(true, GP_SCALED); else APS_G(false, GP_SCALED);
#undef APS_G
}

static void launch_lp_gemm(int variant, bool kahan, int pm, dim3 grid, hipStream_t s, const GemmArgs& g,
                           const FmtK& fi, const FmtK& fa) {
#define APS_LG(v) \
    if (variant == (v)) launch_lp_gemm_v<v>(kahan, pm, grid, s, g, fi, fa);
    APS_LG(0) APS_LG(1) APS_LG(2) APS_LG(3) APS_LG(4) APS_LG(5) APS_LG(6) APS_LG(7) APS_LG(8) APS_LG(9)
#undef APS_LG
}

extern "C" int aps_lp_gemm(const float* A, int64_t lda, const float* B, int64_t ldb, float* C, int64_t ldc,
                           int32_t M, int32_t N, int32_t K, aps_format in_fmt, aps_format acc_fmt,
                           int32_t accumulator, void* stream) {
    if (M < 0 || N < 0 || K < 0 || M > APS_MAX_GEMM_DIM || N > APS_MAX_GEMM_DIM || K > APS_MAX_GEMM_DIM)
        return APS_ERR_SIZE;
    const bool has_out = (int64_t)M * N > 0;
    if (has_out && (!C || (K > 0 && (!A || !B)))) return APS_ERR_NULL;
    if (has_out && (ldc < N || (K > 0 && (lda < K || ldb < N)))) return APS_ERR_SIZE;
    int st = fmt_status(in_fmt);
    if (st != APS_OK) return st;
    st = fmt_status(acc_fmt);
    if (st != APS_OK) return st;
    if (accumulator != APS_ACC_SEQUENTIAL && accumulator != APS_ACC_KAHAN) return APS_ERR_UNSUPPORTED;
    // formats rounded in fp64 (class GEN) are not built into the GEMM
    if (make_fmtk(in_fmt).variant == V_GEN || make_fmtk(acc_fmt).variant == V_GEN) return APS_ERR_UNSUPPORTED;
    // the product of two input values must be exact in fp32, or round to zero anyway
    const int emin_in = 1 - in_fmt.bias, emin_acc = 1 - acc_fmt.bias;
    if (in_fmt.m > 11) return APS_ERR_UNSUPPORTED;
    if (2 * (emin_in - in_fmt.m) < -149 && 2 * (in_fmt.m + 1) > emin_acc - acc_fmt.m + 149) return APS_ERR_UNSUPPORTED;
    if (!has_out) return APS_OK;
    const FmtK fi = make_fmtk(in_fmt), fa = make_fmtk(acc_fmt);
    const int64_t mt = (M + GT - 1) / GT, nt = (N + GT - 1) / GT;
    GemmArgs g{A, B, C, lda, ldb, ldc, M, N, K, 0, 0, mt * nt, (int32_t)nt, 1.0f};
    // Pre-scale the staged operands by 2^ka and 2^kb (ka + kb = k) when both
    // stay below 2^128: a value below 2^(emax_in+1) times 2^(127-emax_in) does.
    const int room = 127 - fi.emax;
    int pm = GP_LDEXP;
    if (fa.k <= 2 * room) {
        g.ka = fa.k < room ? fa.k : room;
        g.kb = fa.k - g.ka;
        pm = GP_SCALED;
        // every product has at most 2(m_in+1) significant bits
        const int cls = fa.variant <= V_INT_M0 ? CLS_INT : (fa.variant <= V_TOP_M0 ? CLS_TOP : CLS_LOW);
        if (cls != CLS_INT && acc_fmt.m > 0 && 2 * (in_fmt.m + 1) <= acc_fmt.m + 1) pm = GP_FIT;
    }
    if (pm == GP_FIT) {
        // GP_GRID where the step's exponent Q is >= 0 (the format spans at
        // most 128 binades with its subnormals, so a staged product overflows
        // fp32 only where the format does) and the operands can carry
        // 2^(m - emin) between them as fp32 normals: staged values from the
        // input's smallest subnormal to below 2^128
        const int q = fa.emin + fa.k - acc_fmt.m;
        const int kq = acc_fmt.m - fa.emin;
        const int lo = -126 - (fi.emin - in_fmt.m), hi = 127 - fi.emax;
        const int ka = std::min(std::max(kq / 2, lo), hi), kb = kq - ka;
        if (q >= 0 && q <= 127 && kb >= lo && kb <= hi) {
            g.ka = ka;
            g.kb = kb;
            g.qs = pow2f_host(q);
            pm = GP_GRID;
        }
    }
    if (pm != GP_LDEXP && acc_fmt.m > 0 && 2 * (in_fmt.m + 1) <= acc_fmt.m + 1 &&
        2 * (fi.emin - in_fmt.m) >= fa.emin) {
        // products staged in the working domain (ka + kb = k, both >= 0, so
        // every staged value stays exact), each one fits and none is
        // subnormal in the accumulator: GP_EXACT
        g.ka = fa.k < room ? fa.k : room;
        g.kb = fa.k - g.ka;
        g.qs = 1.0f;
        pm = (acc_fmt.e == 8 && acc_fmt.m == 7 && acc_fmt.bias == 127) ? GP_BF16 : GP_EXACT;
    }
    const dim3 grid((unsigned)std::min<int64_t>(g.tiles, INT32_MAX));
    // the accumulator is IEEE half and every input value a half (at most 10
    // mantissa bits, at most 2^15 and no finer than half's step 2^-24); such
    // an input format is of class TOP or LOW
    const bool half_acc = acc_fmt.e == 5 && acc_fmt.m == 10 && acc_fmt.bias == 15;
    if (half_acc && in_fmt.m <= 10 && fi.emax <= 15 && fi.emin - in_fmt.m >= -24) {
        const int64_t hmt = (M + HGT - 1) / HGT, hnt = (N + HGT - 1) / HGT;
        g.tiles = hmt * hnt;
        g.ntn = (int32_t)hnt;
        const dim3 hgrid((unsigned)std::min<int64_t>(g.tiles, INT32_MAX));
        const hipStream_t hs = (hipStream_t)stream;
        const bool kh = accumulator == APS_ACC_KAHAN;
#define APS_HK(VI)                                                                          \
    if (input_mode_is((VI), fi)) {                                                              \
        if (kh)                                                                            \
            hipLaunchKernelGGL((k_lp_gemm_h<true, VI>), hgrid, dim3(BLOCK), 0, hs, g, fi);  \
        else                                                                               \
            hipLaunchKernelGGL((k_lp_gemm_h<false, VI>), hgrid, dim3(BLOCK), 0, hs, g, fi); \
        return launched();                                                                 \
    }
        APS_HK(VI_E5M2) APS_HK(VI_E4M3) APS_HK(V_TOP_F32) APS_HK(V_TOP_M0) APS_HK(V_LOW_F32) APS_HK(V_LOW_M0)
#undef APS_HK
        g.tiles = mt * nt;  // another input class: the emulated kernel
        g.ntn = (int32_t)nt;
    }
    launch_lp_gemm(fa.variant, accumulator == APS_ACC_KAHAN, pm, grid, (hipStream_t)stream, g, fi, fa);
    return launched();
}
