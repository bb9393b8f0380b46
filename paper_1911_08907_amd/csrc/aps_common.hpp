// aps_common.hpp -- device code and host helpers shared by the kernel files
// of the APS gradient path on gfx950 (Algorithm 1 of arXiv 1911.08907 for W
// data-parallel workers simulated on one GPU).
//
// Work decomposition.  The flat n-element gradient is cut into chunks of
// CH = 1024 elements; each thread owns 4 consecutive elements (one 16-byte
// load per worker row).  A launch has a measured number of blocks per CU
// (BLOCKS_PER_CU, or a kernel's own; stream_grid below) and each block
// walks a contiguous range of chunks, so the layer of a chunk is found by a
// forward scan from the previous one (scalar loads of the offsets table).
// A chunk may cover several layers; as long as they share one palette entry
// the fast kernels handle it with a per-element scale exponent.  Chunks that
// mix palette entries (only possible with several formats) go to a small
// generic kernel, one block per such chunk.
//
// Nothing here allocates memory; every kernel is enqueued on the caller's
// stream.
#pragma once

#include <algorithm>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "aps.h"
#include "aps_format.hpp"

namespace aps {

#ifndef APS_UNROLL
#define APS_UNROLL 4
#endif
#ifndef APS_BLOCKS_PER_CU
#define APS_BLOCKS_PER_CU 16
#endif
#ifndef APS_MAXABS_BLOCKS_PER_CU
#define APS_MAXABS_BLOCKS_PER_CU 4
#endif
#ifndef APS_MAXABS_UNROLL
#define APS_MAXABS_UNROLL 8
#endif

constexpr int BLOCK = 256;
constexpr int VEC = 4;
constexpr int64_t CH = BLOCK * VEC;
constexpr int UNROLL = APS_UNROLL;                // worker rows per register set (two sets in flight)
constexpr int BLOCKS_PER_CU = APS_BLOCKS_PER_CU;  // launch width of the streaming kernels
constexpr int MAXABS_BLOCKS_PER_CU = APS_MAXABS_BLOCKS_PER_CU;
constexpr int MAXABS_UNROLL = APS_MAXABS_UNROLL;  // worker rows per load batch in k_maxabs

typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2v __attribute__((ext_vector_type(2)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

struct Pal {
    FmtK f[APS_MAX_FORMATS];
};

struct Layers {
    const int64_t* __restrict__ offsets;
    const uint8_t* __restrict__ fmt_idx;
    const int32_t* __restrict__ scale_exp;
    int64_t n;
    int32_t L;
    int32_t n_fmts;
};

// Copy of the palette in LDS, for kernels that index it per lane.
__device__ __forceinline__ void pal_to_lds(const Pal& pal, FmtK* spal) {
    if (threadIdx.x < APS_MAX_FORMATS) spal[threadIdx.x] = pal.f[threadIdx.x];
    __syncthreads();
}

// Read-only tables (offsets, palette indices, scale exponents) are read
// through the constant address space: uniform reads then become scalar loads,
// which do not wait for the kernel's own outstanding vector stores.
template <class T>
__device__ __forceinline__ T cld(const T* p, int64_t i) {
    return ((const __attribute__((address_space(4))) T*)p)[i];
}

// A palette index (one byte) through a scalar load of its aligned 32-bit word.
__device__ __forceinline__ int cld_idx(const uint8_t* p, int64_t i) {
    const uintptr_t a = (uintptr_t)(p + i);
    const uint32_t w = *(const __attribute__((address_space(4))) uint32_t*)(a & ~(uintptr_t)3);
    return (int)((w >> ((a & 3u) * 8u)) & 0xFFu);
}

__device__ __forceinline__ float u2f(uint32_t u) { return __uint_as_float(u); }
__device__ __forceinline__ uint32_t f2u(float f) { return __float_as_uint(f); }

__device__ __forceinline__ int clamp_exp(int32_t ft) {
    // |ft| beyond 400 takes every fp32 value to 0 or INF exactly as 400 does
    return ft < -400 ? -400 : (ft > 400 ? 400 : ft);
}

// ------------------------------------------------------------ rounding

template <int V>
struct VT {
    static constexpr int cls = V == V_GEN ? CLS_GEN : (V <= V_INT_M0 ? CLS_INT : (V <= V_TOP_M0 ? CLS_TOP : CLS_LOW));
    static constexpr int acc = V == V_INT_EXACT ? ACC_EXACT
                               : ((V == V_INT_F64 || V == V_TOP_F64 || V == V_LOW_F64) ? ACC_F64 : ACC_F32);
    static constexpr bool m0 = (V == V_INT_M0 || V == V_TOP_M0 || V == V_LOW_M0);
};

// Class GEN: the format value of v (native, k = 0), rounded in fp64.  Above
// 2^emin the fp64 pattern keeps m mantissa bits, ties to even (m = 0: up, the
// even multiple); below, the magic constant puts v on the subnormal grid
// 2^(emin - m) with fp64's own ties-to-even.  From 2^(emax + 1) up it is INF;
// NaN stays NaN.  The result is a format value, so exact in fp32.
__device__ __forceinline__ float round_gen(double v, const FmtK& f) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint64_t tie = f.m ? ((b >> f.sh64) & 1ull) : 0ull;
    const double rn = __longlong_as_double((long long)((b + f.half64 + tie) & f.mask64));
    const double a = __builtin_fabs(v);
    const double rs = __builtin_copysign((a + f.c064) - f.c064, v);
    double r = (a >= f.thr64) ? rn : rs;
    r = (__builtin_fabs(r) >= f.ovf64) ? __builtin_copysign(__builtin_inf(), v) : r;
    return (float)((v != v) ? v : r);
}

// Working-domain format value of y, a value already in the working domain
// (fl32 of the scaled input).  Sets `bad` when y is NaN (m = 0 formats have
// no NaN pattern that survives the rounding, so NaN is tracked on the side).
template <int V>
__device__ __forceinline__ float quant_w(float y, const FmtK& f, bool& bad) {
    using T = VT<V>;
    if constexpr (T::m0) bad |= (y != y);
    if constexpr (T::cls == CLS_GEN) {
        return round_gen((double)y, f);
    } else if constexpr (T::acc == ACC_EXACT) {
        return y;
    } else if constexpr (T::cls == CLS_INT) {
        const uint32_t b = f2u(y);
        uint32_t r;
        if constexpr (T::m0) {
            // tie bit: 1 for normal fp32 (round half up), 0 on fp32's subnormal grid
            r = b + ((1u << 22) - 1u) + min(__builtin_amdgcn_ubfe(b, 23, 8), 1u);
        } else {
            r = b + f.half + __builtin_amdgcn_ubfe(b, f.sh, T::acc == ACC_F32 ? 1u : f.lsbw);
            r = (y != y) ? b : r;  // a NaN keeps its quiet payload
        }
        return u2f(r & f.mask);
    } else {
        const uint32_t b = f2u(y);
        uint32_t rn;
        if constexpr (T::m0)
            rn = b + f.half;
        else
            rn = b + f.half + __builtin_amdgcn_ubfe(b, f.sh, T::acc == ACC_F32 ? 1u : f.lsbw);
        uint32_t rsb;
        if constexpr (T::cls == CLS_LOW && !T::m0) {
            // on the scale where the subnormal step is 1: an integer, ties to even, sign kept
            rsb = f2u(__builtin_rintf(y * f.qi) * f.qs);
        } else {
            float ys = y;
            if constexpr (T::cls == CLS_LOW) ys = __builtin_amdgcn_ldexpf(y, -f.j);
            float rs = (__builtin_fabsf(ys) + f.c0) - f.c0;
            if constexpr (T::cls == CLS_LOW) rs = __builtin_amdgcn_ldexpf(rs, f.j);
            rsb = (b & 0x80000000u) | f2u(rs);
        }
        // NaN fails the compare and takes the subnormal path, which keeps it NaN
        const uint32_t r = (__builtin_fabsf(y) >= f.thr) ? rn : rsb;
        return u2f(r & f.mask);
    }
}

// Working-domain format value of fl32(x * 2^F) (F already includes the
// domain shift k).
template <int V>
__device__ __forceinline__ float quant(float x, int F, const FmtK& f, bool& bad) {
    return quant_w<V>(__builtin_amdgcn_ldexpf(x, F), f, bad);
}

// quant_w for a y whose significand already fits the format's (at most m+1
// significant bits) and whose overflow is already INF: only the subnormal
// range rounds.  TOP and LOW classes, m >= 1.
template <int V>
__device__ __forceinline__ float quant_fit(float y, const FmtK& f) {
    static_assert((VT<V>::cls == CLS_TOP || VT<V>::cls == CLS_LOW) && !VT<V>::m0, "TOP or LOW class, m >= 1");
    const uint32_t b = f2u(y);
    uint32_t ab = b & 0x7FFFFFFFu;
    asm volatile("" : "+v"(ab));  // keep |y| in a register: two-operand forms below, no abs modifiers
    float ys = u2f(ab);
    if constexpr (VT<V>::cls == CLS_LOW) ys = __builtin_amdgcn_ldexpf(ys, -f.j);
    float rs = (ys + f.c0) - f.c0;
    if constexpr (VT<V>::cls == CLS_LOW) rs = __builtin_amdgcn_ldexpf(rs, f.j);
    // NaN fails the compare and takes the subnormal path, which keeps it NaN
    return (f.thr <= u2f(ab)) ? y : u2f(f2u(rs) | (b & 0x80000000u));
}

// R_fmt(s + q) for two working-domain format values.
template <int V>
__device__ __forceinline__ float accum(float s, float q, const FmtK& f, bool& bad) {
    using T = VT<V>;
    if constexpr (T::cls == CLS_GEN) {
        // the fp64 sum of two fp32 values, rounded to 53 then to m+1 <= 24
        // bits, is the rounded exact sum (53 >= 2 * 24 + 2); below 2^emin the
        // exact sum is a multiple of the subnormal step and exact in fp64
        return round_gen((double)s + (double)q, f);
    } else if constexpr (T::acc == ACC_EXACT) {
        return s + q;
    } else if constexpr (T::acc == ACC_F32) {
        const float t = s + q;
        if constexpr (T::m0) bad |= (t != t);
        const uint32_t b = f2u(t);
        uint32_t r;
        if constexpr (T::m0)
            r = b + f.half;
        else
            r = b + f.half + __builtin_amdgcn_ubfe(b, f.sh, 1u);
        return u2f(r & f.mask);
    } else {
        const double t = (double)s + (double)q;
        const uint64_t b = (uint64_t)__double_as_longlong(t);
        const uint64_t r = (b + f.half64 + ((b >> f.sh64) & 1ull)) & f.mask64;
        return (float)__longlong_as_double((long long)r);
    }
}

template <int V>
__device__ __forceinline__ float finish(float s, bool bad) {
    if constexpr (VT<V>::m0) return bad ? __builtin_nanf("") : s;
    return s;
}

// ---------------------------------------------------------------- codes

// code of a native-domain format value v.  Every case is computed and one is
// selected, so the wave never splits on the value's class.  Where 2^emin is
// an fp32 subnormal (esh > 0) the normal case reads the pattern of v * 2^esh.
__device__ __forceinline__ uint32_t encode(float v, const FmtK& f) {
    const uint32_t b = f2u(v);
    const uint32_t sign = (b >> 31) << (f.e + f.m);
    const uint32_t a = b & 0x7FFFFFFFu;
    // bits of 2^emin (>= 2^-149: emin - m >= -149)
    const uint32_t lo = f.emin >= -126 ? (uint32_t)(f.emin + 127) << 23 : 1u << (f.emin + 149);
    // below 2^emin: the subnormal code counts multiples of 2^(emin-m); the
    // clamp keeps the conversion's input finite when another case is taken
    const uint32_t c_sub = (uint32_t)__builtin_amdgcn_ldexpf(u2f(min(a, lo)), f.m - f.emin);
    const uint32_t an = f2u(__builtin_amdgcn_ldexpf(u2f(a), f.esh));
    const uint32_t c_norm = (an >> (23 - f.m)) - ((uint32_t)(127 + f.esh - f.bias) << f.m);
    const uint32_t c_nan = (uint32_t)f.emax_code | (f.m > 0 ? (1u << (f.m - 1)) : 0u);
    uint32_t c = a < lo ? c_sub : c_norm;
    c = a == 0x7F800000u ? (uint32_t)f.emax_code : c;
    c = a > 0x7F800000u ? c_nan : c;
    return sign | c;
}

__device__ __forceinline__ float decode(uint32_t code, const FmtK& f) {
    const uint32_t ef = (code >> f.m) & ((1u << f.e) - 1u);
    const uint32_t mant = code & ((1u << f.m) - 1u);
    float a;
    if (ef == (1u << f.e) - 1u)
        a = mant ? __builtin_nanf("") : __builtin_inff();
    else if (ef == 0)
        a = __builtin_amdgcn_ldexpf((float)mant, f.emin - f.m);
    else  // built at 2^esh times the value (an fp32 normal), then scaled back exactly
        a = __builtin_amdgcn_ldexpf(u2f(((ef + 127u + (uint32_t)f.esh - (uint32_t)f.bias) << 23) | (mant << (23 - f.m))),
                                    -f.esh);
    return ((code >> (f.e + f.m)) & 1u) ? -a : a;
}

__host__ __device__ __forceinline__ int64_t code_byte(int64_t j, int cls) {
    return cls == 0 ? (j >> 1) : (cls == 1 ? j : 2 * j);
}

// Store the codes of elements j..j+3 (j % 4 == 0) of a row, all four present.
__device__ __forceinline__ void store_codes4_full(uint8_t* row, int64_t j, const uint32_t c[4], int cls) {
    // streaming (non-temporal) stores: the codes are not read back by this launch
    if (cls == 0) {
        const uint16_t v = (uint16_t)((c[0] & 15u) | ((c[1] & 15u) << 4) | ((c[2] & 15u) << 8) | ((c[3] & 15u) << 12));
        __builtin_nontemporal_store(v, (uint16_t*)(row + (j >> 1)));
    } else if (cls == 1) {
        const uint32_t v = (c[0] & 255u) | ((c[1] & 255u) << 8) | ((c[2] & 255u) << 16) | (c[3] << 24);
        __builtin_nontemporal_store(v, (uint32_t*)(row + j));
    } else {
        const u2v v = {(c[0] & 0xFFFFu) | (c[1] << 16), (c[2] & 0xFFFFu) | (c[3] << 16)};
        __builtin_nontemporal_store(v, (u2v*)(row + 2 * j));
    }
}

// Store the codes of elements j..j+3 (j % 4 == 0) of a row; only those < lim.
__device__ __forceinline__ void store_codes4(uint8_t* row, int64_t j, const uint32_t c[4], int cls, int64_t lim) {
    if (j + 4 <= lim) {
        store_codes4_full(row, j, c, cls);
        return;
    }
    for (int e = 0; e < 4; ++e) {
        const int64_t jj = j + e;
        if (jj >= lim) break;
        if (cls == 0) {
            uint8_t* p = row + (jj >> 1);
            const int sh = (int)(jj & 1) * 4;
            *p = (uint8_t)((*p & ~(15u << sh)) | ((c[e] & 15u) << sh));
        } else if (cls == 1) {
            row[jj] = (uint8_t)c[e];
        } else {
            *(uint16_t*)(row + 2 * jj) = (uint16_t)c[e];
        }
    }
}

__device__ __forceinline__ void put_code(uint8_t* row, int64_t j, uint32_t c, int cls) {
    if (cls == 1)
        row[j] = (uint8_t)c;
    else
        *(uint16_t*)(row + 2 * j) = (uint16_t)c;
}

__device__ __forceinline__ uint32_t load_code(const uint8_t* row, int64_t j, int cls) {
    if (cls == 0) return (row[j >> 1] >> ((j & 1) * 4)) & 15u;
    if (cls == 1) return row[j];
    return *(const uint16_t*)(row + 2 * j);
}

// --------------------------------------------------------- chunk walking

// Largest i in [0, L-1] with offsets[i] <= pos (pos < n), searching from a hint.
__device__ __forceinline__ int find_layer(const int64_t* __restrict__ off, int L, int64_t pos, int hint) {
    int i = hint;
    if (cld(off, i) > pos) {
        int lo = 0, hi = i;
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (cld(off, mid) <= pos) lo = mid; else hi = mid;
        }
        return lo;
    }
    for (int s = 0; s < 4; ++s) {
        if (i + 1 >= L || cld(off, i + 1) > pos) return i;
        ++i;
    }
    int lo = i, hi = L;  // off[lo] <= pos; off[L] = n > pos
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (cld(off, mid) <= pos) lo = mid; else hi = mid;
    }
    return lo;
}

// Layers of chunk [start, end): first i0, last i1 (uniform); whether they all
// use one palette entry, and which.
struct ChunkInfo {
    int i0, i1, pidx;
    bool mixed;
};

__device__ __forceinline__ ChunkInfo chunk_layers(const Layers& ly, int64_t start, int64_t end, int hint) {
    ChunkInfo ci;
    ci.i0 = find_layer(ly.offsets, ly.L, start, hint);
    int i = ci.i0;
    while (cld(ly.offsets, i + 1) < end) ++i;  // offsets[L] = n >= end
    ci.i1 = i;
    ci.pidx = ly.fmt_idx ? cld_idx(ly.fmt_idx, ci.i0) : 0;
    ci.mixed = false;
    if (ly.fmt_idx && ci.i1 > ci.i0) {
        for (int t = ci.i0 + 1; t <= ci.i1; ++t) {
            if (cld(ly.offsets, t) == cld(ly.offsets, t + 1)) continue;  // empty layer
            if (cld_idx(ly.fmt_idx, t) != ci.pidx) ci.mixed = true;
        }
    }
    return ci;
}

// Per-element scale exponent for elements j..j+3 of a chunk spanning layers i0..i1.
__device__ __forceinline__ void elem_scales(const Layers& ly, const ChunkInfo& ci, int64_t j, int32_t ft[4]) {
    int li = ci.i0;
    for (int e = 0; e < 4; ++e) {
        const int64_t jj = j + e;
        while (li < ci.i1 && ly.offsets[li + 1] <= jj) ++li;
        ft[e] = ly.scale_exp ? clamp_exp(ly.scale_exp[li]) : 0;
    }
}

__device__ __forceinline__ void block_range(int64_t nitems, int64_t& b, int64_t& e) {
    const int64_t G = gridDim.x;
    b = nitems * (int64_t)blockIdx.x / G;
    e = nitems * ((int64_t)blockIdx.x + 1) / G;
}

__device__ __forceinline__ f4 ld4(const float* p) { return __builtin_nontemporal_load((const f4*)p); }

// ======================================================== K1: max-abs

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    for (int o = 32; o > 0; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o, 64));
    return v;
}

// Block-wide max of v (all threads call it), then one atomicMax if nonzero.
__device__ __forceinline__ void block_max_atomic(uint32_t v, uint32_t* dst, uint32_t* red) {
    v = wave_max_u32(v);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = red[0];
        for (int k = 1; k < BLOCK / 64; ++k) t = max(t, red[k]);
        if (t) atomicMax(dst, t);
    }
    __syncthreads();
}

// ========================================================= K2: scales

__device__ __forceinline__ int ceil_log2_bits(uint32_t t) {
    // t: bits of a finite positive fp32
    const uint32_t ef = t >> 23, frac = t & 0x7FFFFFu;
    if (ef == 0) {  // subnormal: t = frac * 2^-149
        const int fl = 31 - __builtin_clz(frac);
        return fl - 149 + ((frac & (frac - 1u)) ? 1 : 0);
    }
    return (int)ef - 127 + (frac ? 1 : 0);
}

// ========================================================= row streaming

// Makes the compiler wait for the load that produced v here, without an
// instruction: an empty asm that reads its registers.
__device__ __forceinline__ void touch(const f4& v) { asm volatile("" ::"v"(v.x), "v"(v.y), "v"(v.z), "v"(v.w)); }

// Streams W rows of one thread's 16-byte column slice through the callbacks:
// first(row 0), then step(row w, valid) for w = 1, 2, ... in order.  Two
// register sets of U rows (UNROLL by default) are in flight: while one set is
// consumed, the loads of the next U rows are outstanding; the scheduling barrier keeps
// those loads ahead of the math.  Rows past W-1 are loaded from row W-1 and
// handed to step() with valid = false, so every path issues the same loads
// and the compiler waits for exactly the row it is about to use.
// after_issue() runs once, right after the first 2*UNROLL loads are issued.
//
// The sets of UNROLL rows are numbered 0 .. nsets-1.  Set 0 and set 1 are
// loaded up front; a full step consumes set s (all rows valid) after issuing
// the loads of set s+1, for s = 1 .. nsets-2; the last set is consumed with
// per-row validity.  The full steps run as a counted loop of pairs with no
// exit in its body: an exit in the middle of the body is merged by the
// compiler's control-flow structurizer into the back edge, and the loads it
// would leave outstanding then force waits at the top of every iteration.
template <int U = UNROLL, class Load, class AfterIssue, class First, class Step>
__device__ __forceinline__ void stream_rows(int W, Load load, AfterIssue after_issue, First first, Step step) {
    f4 A[U], B[U];
#pragma unroll
    for (int u = 0; u < U; ++u) A[u] = load(min(u, W - 1));
#pragma unroll
    for (int u = 0; u < U; ++u) B[u] = load(min(U + u, W - 1));
    __builtin_amdgcn_sched_barrier(0);
    after_issue();
    first(A[0]);
    const int nsets = (W + U - 1) / U;
    if (nsets == 1) {
#pragma unroll
        for (int u = 1; u < U; ++u) {
            touch(A[u]);
            step(A[u], u < W);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            touch(B[u]);
            step(B[u], false);
        }
        return;
    }
#pragma unroll
    for (int u = 1; u < U; ++u) step(A[u], true);
    int w = U;  // first row of the set being consumed
#define APS_FULL(CUR, NXT)                                                \
    {                                                                     \
        _Pragma("unroll") for (int u = 0; u < U; ++u)                     \
            NXT[u] = load(min(w + U + u, W - 1));                         \
        __builtin_amdgcn_sched_barrier(0);                                \
        _Pragma("unroll") for (int u = 0; u < U; ++u) step(CUR[u], true); \
        w += U;                                                           \
    }
#define APS_LAST(CUR)                                     \
    {                                                     \
        _Pragma("unroll") for (int u = 0; u < U; ++u) {   \
            touch(CUR[u]);                                \
            step(CUR[u], w + u < W);                      \
        }                                                 \
    }
    const int nfull = nsets - 2;
#pragma unroll 1
    for (int it = 0; it < nfull / 2; ++it) {
        APS_FULL(B, A)
        APS_FULL(A, B)
    }
    if (nfull & 1) {
        APS_FULL(B, A)
        APS_LAST(A)
    } else {
        APS_LAST(B)
    }
#undef APS_FULL
#undef APS_LAST
}

// ===================================================== K4: sim reduce

struct ReduceArgs {
    const float* __restrict__ G;
    float* __restrict__ out;
    uint8_t* __restrict__ codes;
    int64_t ld;
    int32_t W;
    uint32_t flags;
    int32_t code_cls;
};

// A thread's finished outputs (4 elements), kept in registers until the next
// chunk's first loads have been issued.  Loads and stores share one in-order
// completion counter, so a store issued before those loads would make the
// first wait for them also wait for the store's write acknowledgement.
struct PendingOut {
    f4 o;
    uint32_t c[4];
    int64_t j, lim;  // first element; elements >= lim are not written
    bool valid;
};

__device__ __forceinline__ void flush_out(const ReduceArgs& a, PendingOut& pd) {
    if (!pd.valid) return;
    pd.valid = false;
    if (a.out) {
        const int64_t j = pd.j, lim = pd.lim;
        if (j + 4 <= lim) {
            __builtin_nontemporal_store(pd.o, (f4*)(a.out + j));
        } else {
            if (j < lim) a.out[j] = pd.o.x;
            if (j + 1 < lim) a.out[j + 1] = pd.o.y;
            if (j + 2 < lim) a.out[j + 2] = pd.o.z;
        }
    }
    if (a.codes) store_codes4(a.codes, pd.j, pd.c, a.code_cls, pd.lim);
}

// Finished fp32 outputs waiting in LDS, each thread in its own slots (no
// other thread reads them, so no barrier), written OUT_STAGE chunks at a
// time or when the block is done: writes in the middle of the row reads cost
// the streaming kernels more than their bytes, and fewer, larger bursts of
// them cost less.  For outputs without codes.
constexpr int OUT_STAGE = 6;

struct OutStage {
    f4* o;        // [OUT_STAGE][BLOCK]
    int32_t* j;   // first element (n <= 2^30)
    int32_t* lim; // elements >= lim are not written
    int cnt;      // this thread's filled slots
};

__device__ __forceinline__ void drain_out(const ReduceArgs& a, OutStage& st) {
    const int t = threadIdx.x;
    for (int s = 0; s < st.cnt; ++s) {
        const int64_t j = st.j[s * BLOCK + t], lim = st.lim[s * BLOCK + t];
        const f4 o = st.o[s * BLOCK + t];
        if (j + 4 <= lim) {
            __builtin_nontemporal_store(o, (f4*)(a.out + j));
        } else {
            if (j < lim) a.out[j] = o.x;
            if (j + 1 < lim) a.out[j + 1] = o.y;
            if (j + 2 < lim) a.out[j + 2] = o.z;
        }
    }
    st.cnt = 0;
}

// Moves the pending record into the stage.  The caller drains a full stage
// between chunks (drain_if_full), outside the row loop.
__device__ __forceinline__ void stage_out(PendingOut& pd, OutStage& st) {
    if (!pd.valid) return;
    pd.valid = false;
    const int t = threadIdx.x;
    st.o[st.cnt * BLOCK + t] = pd.o;
    st.j[st.cnt * BLOCK + t] = (int32_t)pd.j;
    st.lim[st.cnt * BLOCK + t] = (int32_t)pd.lim;
    ++st.cnt;
}

__device__ __forceinline__ void drain_if_full(const ReduceArgs& a, OutStage& st) {
    if (st.cnt == OUT_STAGE) drain_out(a, st);
}


// The fused scale + cast + rounded sum + unscale of 4 consecutive elements
// over the W rows.  With MAX it also returns the largest |x| bit pattern of
// each of the 4 columns in mx (rows past the end read as -0: no effect).
// With a stage (no codes), the previous chunk's outputs go to it instead of
// straight to memory; the stage must have a free slot (drain_if_full).
template <int V, bool MAX = false>
__device__ __forceinline__ void reduce_vec(const ReduceArgs& a, const FmtK& f, int64_t j, int64_t lim,
                                           const int32_t ft[4], PendingOut& pd, uint32_t* mx = nullptr,
                                           OutStage* st = nullptr) {
    const bool inq = a.flags & APS_INPUT_QUANTIZED;
    const bool outs = a.flags & APS_OUTPUT_SCALED;
    int F[4], Fo[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        F[e] = (inq ? 0 : ft[e]) + f.k;
        Fo[e] = -((outs ? 0 : ft[e]) + f.k);
    }
    bool bad0 = false, bad1 = false, bad2 = false, bad3 = false;
    const float* p = a.G + j;
    const int64_t ld = a.ld;
    float s0, s1, s2, s3;
    uint32_t m0 = 0, m1 = 0, m2 = 0, m3 = 0;
    // a row past the last one counts as -0, which leaves every sum unchanged
    // (s + -0 == s, signs of zero included)
    const f4 neg0 = {-0.0f, -0.0f, -0.0f, -0.0f};
    stream_rows(
        a.W, [&](int r) { return ld4(p + (int64_t)r * ld); },
        [&]() {  // the previous chunk's outputs, behind this chunk's loads
            if (st)
                stage_out(pd, *st);
            else
                flush_out(a, pd);
        },
        [&](const f4& x) {
            if constexpr (MAX) {
                m0 = f2u(x.x) & 0x7FFFFFFFu;
                m1 = f2u(x.y) & 0x7FFFFFFFu;
                m2 = f2u(x.z) & 0x7FFFFFFFu;
                m3 = f2u(x.w) & 0x7FFFFFFFu;
            }
            s0 = quant<V>(x.x, F[0], f, bad0);
            s1 = quant<V>(x.y, F[1], f, bad1);
            s2 = quant<V>(x.z, F[2], f, bad2);
            s3 = quant<V>(x.w, F[3], f, bad3);
        },
        [&](const f4& r, bool valid) {
            const f4 v = valid ? r : neg0;
            if constexpr (MAX) {
                m0 = max(m0, f2u(v.x) & 0x7FFFFFFFu);
                m1 = max(m1, f2u(v.y) & 0x7FFFFFFFu);
                m2 = max(m2, f2u(v.z) & 0x7FFFFFFFu);
                m3 = max(m3, f2u(v.w) & 0x7FFFFFFFu);
            }
            s0 = accum<V>(s0, quant<V>(v.x, F[0], f, bad0), f, bad0);
            s1 = accum<V>(s1, quant<V>(v.y, F[1], f, bad1), f, bad1);
            s2 = accum<V>(s2, quant<V>(v.z, F[2], f, bad2), f, bad2);
            s3 = accum<V>(s3, quant<V>(v.w, F[3], f, bad3), f, bad3);
        });
    if constexpr (MAX) {
        mx[0] = m0;
        mx[1] = m1;
        mx[2] = m2;
        mx[3] = m3;
    }
    s0 = finish<V>(s0, bad0);
    s1 = finish<V>(s1, bad1);
    s2 = finish<V>(s2, bad2);
    s3 = finish<V>(s3, bad3);
    pd.o.x = __builtin_amdgcn_ldexpf(s0, Fo[0]);
    pd.o.y = __builtin_amdgcn_ldexpf(s1, Fo[1]);
    pd.o.z = __builtin_amdgcn_ldexpf(s2, Fo[2]);
    pd.o.w = __builtin_amdgcn_ldexpf(s3, Fo[3]);
    if (a.codes) {
        pd.c[0] = encode(__builtin_amdgcn_ldexpf(s0, -f.k), f);
        pd.c[1] = encode(__builtin_amdgcn_ldexpf(s1, -f.k), f);
        pd.c[2] = encode(__builtin_amdgcn_ldexpf(s2, -f.k), f);
        pd.c[3] = encode(__builtin_amdgcn_ldexpf(s3, -f.k), f);
    }
    pd.j = j;
    pd.lim = lim;
    pd.valid = true;
}

// ------------------------------------------------ chains of rounded adds

// R_fmt(a + b) with a NaN sum kept as NaN in the value itself (the rounding
// of an m = 0 format does not keep NaN bit patterns; accum() flags them).
template <int V>
__device__ __forceinline__ float accum_nan(float a, float b, const FmtK& f) {
    bool unused = false;
    const float r = accum<V>(a, b, f, unused);
    if constexpr (VT<V>::m0) {
        const float t = a + b;
        return (t != t) ? t : r;
    }
    return r;
}

// One add of a chain, plain (s = R(s + x)) or Kahan's compensated summation
// with every intermediate rounded to the format.  In the plain chain a NaN
// partial sum stays NaN to the end, so one flag per chain is exact; in Kahan's
// the compensation can turn NaN (INF - INF) while the sum does not, so there
// NaN travels in the values.  `bad` still marks NaN inputs of m = 0 formats.
template <int V, bool KAHAN>
__device__ __forceinline__ void chain_step(float& s, float& c, float x, const FmtK& f, bool& bad) {
    if constexpr (KAHAN) {
        const float y = accum_nan<V>(x, -c, f);
        const float t = accum_nan<V>(s, y, f);
        c = accum_nan<V>(accum_nan<V>(t, -s, f), -y, f);
        s = t;
    } else {
        s = accum<V>(s, x, f, bad);
    }
}

// --------------------------------------------------- one element, any format

// Native-domain value of x cast to the format (scale exponent F includes k);
// an m = 0 format keeps a NaN input NaN.
template <int V>
__device__ __forceinline__ float quant_native(float x, int F, const FmtK& f) {
    bool bad = false;
    const float v = __builtin_amdgcn_ldexpf(quant<V>(x, F, f, bad), -f.k);
    if constexpr (VT<V>::m0) return (x != x) ? x : v;
    return v;
}

// The ragged end of the gradient (fewer than 4 elements left for a thread):
// every row, element by element.
__device__ inline float quant_any(float x, int F, const FmtK& f) {
    switch (f.variant) {
        case V_INT_F32: return quant_native<V_INT_F32>(x, F, f);
        case V_INT_F64: return quant_native<V_INT_F64>(x, F, f);
        case V_INT_EXACT: return quant_native<V_INT_EXACT>(x, F, f);
        case V_INT_M0: return quant_native<V_INT_M0>(x, F, f);
        case V_TOP_F32: return quant_native<V_TOP_F32>(x, F, f);
        case V_TOP_F64: return quant_native<V_TOP_F64>(x, F, f);
        case V_TOP_M0: return quant_native<V_TOP_M0>(x, F, f);
        case V_LOW_F32: return quant_native<V_LOW_F32>(x, F, f);
        case V_LOW_F64: return quant_native<V_LOW_F64>(x, F, f);
        case V_GEN: return quant_native<V_GEN>(x, F, f);
        default: return quant_native<V_LOW_M0>(x, F, f);
    }
}

// One element through the whole W-worker loop, any variant (per-lane format).
template <int V>
__device__ float reduce_elem(const ReduceArgs& a, const FmtK& f, int64_t j, int F) {
    bool bad = false;
    float s = quant<V>(a.G[j], F, f, bad);
    for (int w = 1; w < a.W; ++w) s = accum<V>(s, quant<V>(a.G[(int64_t)w * a.ld + j], F, f, bad), f, bad);
    return finish<V>(s, bad);
}

__device__ inline float reduce_elem_any(const ReduceArgs& a, const FmtK& f, int64_t j, int F) {
    switch (f.variant) {
        case V_INT_F32: return reduce_elem<V_INT_F32>(a, f, j, F);
        case V_INT_F64: return reduce_elem<V_INT_F64>(a, f, j, F);
        case V_INT_EXACT: return reduce_elem<V_INT_EXACT>(a, f, j, F);
        case V_INT_M0: return reduce_elem<V_INT_M0>(a, f, j, F);
        case V_TOP_F32: return reduce_elem<V_TOP_F32>(a, f, j, F);
        case V_TOP_F64: return reduce_elem<V_TOP_F64>(a, f, j, F);
        case V_TOP_M0: return reduce_elem<V_TOP_M0>(a, f, j, F);
        case V_LOW_F32: return reduce_elem<V_LOW_F32>(a, f, j, F);
        case V_LOW_F64: return reduce_elem<V_LOW_F64>(a, f, j, F);
        case V_GEN: return reduce_elem<V_GEN>(a, f, j, F);
        default: return reduce_elem<V_LOW_M0>(a, f, j, F);
    }
}

// Chunks whose layers use different palette entries.  One block per layer
// boundary; the block owning the first boundary strictly inside a chunk
// processes that chunk element by element.
__device__ __forceinline__ bool mixed_chunk_of_boundary(const Layers& ly, int b, int64_t& start, int64_t& end) {
    if (b < 1 || b >= ly.L) return false;
    const int64_t p = cld(ly.offsets, b);
    if (p <= 0 || p >= ly.n || p % CH == 0) return false;
    const int64_t c = p / CH;
    start = c * CH;
    end = min(start + CH, ly.n);
    if (cld(ly.offsets, b - 1) > start) return false;  // an earlier boundary owns it
    const ChunkInfo ci = chunk_layers(ly, start, end, 0);
    return ci.mixed;
}

// ================================================================ host

static inline int device_cus() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    return cus;
}

static inline int64_t grid_for(int64_t items, int per_cu) {
    const int cus = device_cus();
    int64_t g = (int64_t)(cus > 0 ? cus : 256) * per_cu;
    if (g > items) g = items;
    return g < 1 ? 1 : g;
}

// Grid of a streaming kernel over nchunks chunks of W rows: base_per_cu
// blocks per CU, except with few rows (W < 64) on large sets (2^17 chunks or
// more), which run fastest in blocks of about 2.5 chunks each, at most 512
// per CU (measured on MI355X on BERT-large-sized sets at W = 8).
static inline int64_t stream_grid(int64_t nchunks, int32_t W, int base_per_cu) {
    int per_cu = base_per_cu;
    if (W < 64 && nchunks >= ((int64_t)1 << 17)) {
        const int dc = device_cus();
        const int64_t cus = dc > 0 ? dc : 256;
        per_cu = (int)std::min<int64_t>(512, nchunks * 2 / (cus * 5));
    }
    return grid_for(nchunks, per_cu);
}

static inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

static inline int check_palette(const aps_format* fmts, int32_t n_fmts, Pal& pal, int* ccls) {
    if (!fmts) return APS_ERR_NULL;
    if (n_fmts < 1 || n_fmts > APS_MAX_FORMATS) return APS_ERR_SIZE;
    int cls = -1;
    bool mixed_cls = false;
    for (int i = 0; i < n_fmts; ++i) {
        const int st = fmt_status(fmts[i]);
        if (st != APS_OK) return st;
        pal.f[i] = make_fmtk(fmts[i]);
        const int c = code_class(pal.f[i].code_bits);
        if (cls >= 0 && c != cls) mixed_cls = true;
        cls = c;
    }
    for (int i = n_fmts; i < APS_MAX_FORMATS; ++i) pal.f[i] = pal.f[0];
    if (ccls) *ccls = mixed_cls ? -1 : cls;
    return APS_OK;
}

static inline int check_rows(const void* G, int32_t W, int64_t ld, int64_t n, const int64_t* offsets, int32_t L) {
    if (!G || !offsets) return APS_ERR_NULL;
    if (W < 1 || W > APS_MAX_WORKERS || L < 1 || n < 0 || n > APS_MAX_ELEMS || ld < n) return APS_ERR_SIZE;
    if (!aligned16(G) || (ld & 3)) return APS_ERR_ALIGN;
    return APS_OK;
}

static inline int launched() { return hipGetLastError() == hipSuccess ? APS_OK : APS_ERR_DEVICE; }

// which variants occur in the palette
static inline unsigned variant_mask(const Pal& pal, int32_t n_fmts) {
    unsigned m = 0;
    for (int i = 0; i < n_fmts; ++i) m |= 1u << pal.f[i].variant;
    return m;
}

}  // namespace aps

// The kernels are templates over the variant; dispatch table per entry point.
#define APS_FOR_VARIANTS(X) X(0) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10)
