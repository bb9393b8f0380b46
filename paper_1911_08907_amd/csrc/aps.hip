// aps.hip -- HIP kernels (gfx950) and the C ABI of the APS gradient path.
//
// Algorithm 1 of arXiv 1911.08907 for W data-parallel workers simulated on
// one GPU: per-layer max magnitude (FindMaxExp input + AllReduce MAX),
// power-of-two scale exponents (Sec. 3.3.3), scale + cast to a custom float
// (Sec. 3.3.1, Sec. 4), the SUM all-reduce with a low-precision accumulator
// rounded after every add in worker order (Sec. 5), cast back and unscale.
//
// Work decomposition.  The flat n-element gradient is cut into chunks of
// CH = 1024 elements; each thread owns 4 consecutive elements (one 16-byte
// load per worker row).  A launch has about 8 blocks per CU and each block
// walks a contiguous range of chunks, so the layer of a chunk is found by a
// forward scan from the previous one (scalar loads of the offsets table).
// A chunk may cover several layers; as long as they share one palette entry
// the fast kernels handle it with a per-element scale exponent.  Chunks that
// mix palette entries (only possible with several formats) go to a small
// generic kernel, one block per such chunk.
//
// Nothing here allocates memory; every kernel is enqueued on the caller's
// stream.
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
    static constexpr int cls = V <= V_INT_M0 ? CLS_INT : (V <= V_TOP_M0 ? CLS_TOP : CLS_LOW);
    static constexpr int acc = V == V_INT_EXACT ? ACC_EXACT
                               : ((V == V_INT_F64 || V == V_TOP_F64 || V == V_LOW_F64) ? ACC_F64 : ACC_F32);
    static constexpr bool m0 = (V == V_INT_M0 || V == V_TOP_M0 || V == V_LOW_M0);
};

// Working-domain format value of y, a value already in the working domain
// (fl32 of the scaled input).  Sets `bad` when y is NaN (m = 0 formats have
// no NaN pattern that survives the rounding, so NaN is tracked on the side).
template <int V>
__device__ __forceinline__ float quant_w(float y, const FmtK& f, bool& bad) {
    using T = VT<V>;
    if constexpr (T::m0) bad |= (y != y);
    if constexpr (T::acc == ACC_EXACT) {
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
        float ys = y;
        if constexpr (T::cls == CLS_LOW) ys = __builtin_amdgcn_ldexpf(y, -f.j);
        float rs = (__builtin_fabsf(ys) + f.c0) - f.c0;
        if constexpr (T::cls == CLS_LOW) rs = __builtin_amdgcn_ldexpf(rs, f.j);
        const uint32_t rsb = (b & 0x80000000u) | f2u(rs);
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
    static_assert(VT<V>::cls != CLS_INT && !VT<V>::m0, "TOP or LOW class, m >= 1");
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
    if constexpr (T::acc == ACC_EXACT) {
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
// selected, so the wave never splits on the value's class.
__device__ __forceinline__ uint32_t encode(float v, const FmtK& f) {
    const uint32_t b = f2u(v);
    const uint32_t sign = (b >> 31) << (f.e + f.m);
    const uint32_t a = b & 0x7FFFFFFFu;
    const uint32_t lo = (uint32_t)(f.emin + 127) << 23;  // bits of 2^emin
    // below 2^emin: the subnormal code counts multiples of 2^(emin-m); the
    // clamp keeps the conversion's input finite when another case is taken
    const uint32_t c_sub = (uint32_t)__builtin_amdgcn_ldexpf(u2f(min(a, lo)), f.m - f.emin);
    const uint32_t c_norm = (a >> (23 - f.m)) - ((uint32_t)(127 - f.bias) << f.m);
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
    else
        a = u2f(((ef + 127u - (uint32_t)f.bias) << 23) | (mant << (23 - f.m)));
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

// ============================================================ K0: fill

__global__ void k_fill_u32(uint32_t* __restrict__ p, int64_t cnt, uint32_t v) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < cnt) p[i] = v;
}

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

__global__ __launch_bounds__(BLOCK) void k_maxabs(const float* __restrict__ G, int32_t W, int64_t ld,
                                                 Layers ly, uint32_t* __restrict__ maxabs) {
    __shared__ uint32_t red[BLOCK / 64];
    const int64_t nchunks = (ly.n + CH - 1) / CH;
    int64_t cb, ce;
    block_range(nchunks, cb, ce);
    int hint = 0;
    uint32_t run = 0;      // running max for layer run_layer (uniform layer runs only)
    int run_layer = -1;
    for (int64_t c = cb; c < ce; ++c) {
        const int64_t start = c * CH;
        const int64_t end = min(start + CH, ly.n);
        const ChunkInfo ci = chunk_layers(ly, start, end, hint);
        hint = ci.i0;
        const int64_t j = start + (int64_t)threadIdx.x * VEC;
        uint32_t m0 = 0, m1 = 0, m2 = 0, m3 = 0;
        if (j < end) {
            const float* p = G + j;
            // batches of MAXABS_UNROLL rows; rows past W-1 re-read row W-1,
            // which leaves a maximum unchanged
            for (int w = 0; w < W; w += MAXABS_UNROLL) {
                f4 x[MAXABS_UNROLL];
#pragma unroll
                for (int u = 0; u < MAXABS_UNROLL; ++u) x[u] = ld4(p + (int64_t)min(w + u, W - 1) * ld);
#pragma unroll
                for (int u = 0; u < MAXABS_UNROLL; ++u) {
                    m0 = max(m0, f2u(x[u].x) & 0x7FFFFFFFu);
                    m1 = max(m1, f2u(x[u].y) & 0x7FFFFFFFu);
                    m2 = max(m2, f2u(x[u].z) & 0x7FFFFFFFu);
                    m3 = max(m3, f2u(x[u].w) & 0x7FFFFFFFu);
                }
            }
            // elements past the end of the gradient (row padding) do not count
            if (j + 1 >= end) m1 = 0;
            if (j + 2 >= end) m2 = 0;
            if (j + 3 >= end) m3 = 0;
        }
        if (ci.i0 == ci.i1) {
            uint32_t v = max(max(m0, m1), max(m2, m3));
            if (ci.i0 != run_layer) {
                if (run_layer >= 0) block_max_atomic(run, maxabs + run_layer, red);
                run_layer = ci.i0;
                run = 0;
            }
            run = max(run, v);
        } else {
            // chunk crosses layer boundaries: one block-wide max per layer
            const uint32_t mv[4] = {m0, m1, m2, m3};
            for (int li = ci.i0; li <= ci.i1; ++li) {
                const int64_t lo = cld(ly.offsets, li), hi = cld(ly.offsets, li + 1);
                uint32_t v = 0;
                if (j < end)
                    for (int e = 0; e < 4; ++e)
                        if (j + e >= lo && j + e < hi) v = max(v, mv[e]);
                block_max_atomic(v, maxabs + li, red);
            }
        }
    }
    if (run_layer >= 0) block_max_atomic(run, maxabs + run_layer, red);
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

__global__ void k_scales(const uint32_t* __restrict__ maxabs, int32_t L, int32_t N, Pal pal,
                         const uint8_t* __restrict__ fmt_idx, int32_t* __restrict__ scale_exp) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= L) return;
    const FmtK& f = spal[fmt_idx ? fmt_idx[i] : 0];
    const uint32_t gb = maxabs[i] & 0x7FFFFFFFu;
    int32_t r = 0;
    if (gb != 0 && gb < 0x7F800000u) {
        const float t = (float)N * u2f(gb);  // fl32(N * ghat), N <= 2^24 is exact in fp32
        const uint32_t tb = f2u(t);
        if (tb < 0x7F800000u) r = f.emax - ceil_log2_bits(tb);
    }
    scale_exp[i] = r;
}

// ========================================================= row streaming

// Makes the compiler wait for the load that produced v here, without an
// instruction: an empty asm that reads its registers.
__device__ __forceinline__ void touch(const f4& v) { asm volatile("" ::"v"(v.x), "v"(v.y), "v"(v.z), "v"(v.w)); }

// Streams W rows of one thread's 16-byte column slice through the callbacks:
// first(row 0), then step(row w, valid) for w = 1, 2, ... in order.  Two
// register sets of UNROLL rows are in flight: while one set is consumed, the
// loads of the next UNROLL rows are outstanding; the scheduling barrier keeps
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
template <class Load, class AfterIssue, class First, class Step>
__device__ __forceinline__ void stream_rows(int W, Load load, AfterIssue after_issue, First first, Step step) {
    f4 A[UNROLL], B[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) A[u] = load(min(u, W - 1));
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) B[u] = load(min(UNROLL + u, W - 1));
    __builtin_amdgcn_sched_barrier(0);
    after_issue();
    first(A[0]);
    const int nsets = (W + UNROLL - 1) / UNROLL;
    if (nsets == 1) {
#pragma unroll
        for (int u = 1; u < UNROLL; ++u) {
            touch(A[u]);
            step(A[u], u < W);
        }
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            touch(B[u]);
            step(B[u], false);
        }
        return;
    }
#pragma unroll
    for (int u = 1; u < UNROLL; ++u) step(A[u], true);
    int w = UNROLL;  // first row of the set being consumed
#define APS_FULL(CUR, NXT)                                                     \
    {                                                                          \
        _Pragma("unroll") for (int u = 0; u < UNROLL; ++u)                     \
            NXT[u] = load(min(w + UNROLL + u, W - 1));                         \
        __builtin_amdgcn_sched_barrier(0);                                     \
        _Pragma("unroll") for (int u = 0; u < UNROLL; ++u) step(CUR[u], true); \
        w += UNROLL;                                                           \
    }
#define APS_LAST(CUR)                                                          \
    {                                                                          \
        _Pragma("unroll") for (int u = 0; u < UNROLL; ++u) {                   \
            touch(CUR[u]);                                                     \
            step(CUR[u], w + u < W);                                           \
        }                                                                      \
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

template <int V>
__device__ __forceinline__ void reduce_vec(const ReduceArgs& a, const FmtK& f, int64_t j, int64_t lim,
                                           const int32_t ft[4], PendingOut& pd) {
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
    // a row past the last one counts as -0, which leaves every sum unchanged
    // (s + -0 == s, signs of zero included)
    const f4 neg0 = {-0.0f, -0.0f, -0.0f, -0.0f};
    stream_rows(
        a.W, [&](int r) { return ld4(p + (int64_t)r * ld); },
        [&]() { flush_out(a, pd); },  // the previous chunk's outputs, behind this chunk's loads
        [&](const f4& x) {
            s0 = quant<V>(x.x, F[0], f, bad0);
            s1 = quant<V>(x.y, F[1], f, bad1);
            s2 = quant<V>(x.z, F[2], f, bad2);
            s3 = quant<V>(x.w, F[3], f, bad3);
        },
        [&](const f4& r, bool valid) {
            const f4 v = valid ? r : neg0;
            s0 = accum<V>(s0, quant<V>(v.x, F[0], f, bad0), f, bad0);
            s1 = accum<V>(s1, quant<V>(v.y, F[1], f, bad1), f, bad1);
            s2 = accum<V>(s2, quant<V>(v.z, F[2], f, bad2), f, bad2);
            s3 = accum<V>(s3, quant<V>(v.w, F[3], f, bad3), f, bad3);
        });
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

template <int V>
__global__ __launch_bounds__(BLOCK) void k_sim_reduce(ReduceArgs a, Layers ly, Pal pal) {
    const int64_t nchunks = (ly.n + CH - 1) / CH;
    int64_t cb, ce;
    block_range(nchunks, cb, ce);
    int hint = 0;
    PendingOut pd;
    pd.valid = false;
    for (int64_t c = cb; c < ce; ++c) {
        const int64_t start = c * CH;
        const int64_t end = min(start + CH, ly.n);
        const ChunkInfo ci = chunk_layers(ly, start, end, hint);
        hint = ci.i0;
        if (ci.mixed) continue;  // handled by k_sim_reduce_mixed
        const FmtK& f = pal.f[ci.pidx];
        if (f.variant != V) continue;  // another launch owns this format
        const int64_t j = start + (int64_t)threadIdx.x * VEC;
        if (j >= end) continue;
        int32_t ft[4];
        if (ci.i0 == ci.i1) {
            const int32_t t = ly.scale_exp ? clamp_exp(cld(ly.scale_exp, ci.i0)) : 0;
            ft[0] = ft[1] = ft[2] = ft[3] = t;
        } else {
            elem_scales(ly, ci, j, ft);
        }
        reduce_vec<V>(a, f, j, end, ft, pd);
    }
    flush_out(a, pd);
}

// ======================================= K4x: summation orders, Kahan

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

struct Order {
    int32_t log2k;  // group size k = 2^log2k
    int32_t ng;     // number of groups W / k
};

// Worker of the r-th add for an element of ring segment seg: the groups in
// master order seg, seg+1, ... (mod ng), each in worker order.
__device__ __forceinline__ int order_row(int r, int seg, const Order& od) {
    int g = seg + (r >> od.log2k);
    if (g >= od.ng) g -= od.ng;
    return (g << od.log2k) + (r & ((1 << od.log2k) - 1));
}

template <int V, bool KAHAN>
__device__ __forceinline__ void reduce_vec_ex(const ReduceArgs& a, const FmtK& f, int64_t j, int64_t lim,
                                              const int32_t ft[4], int seg, const Order& od, PendingOut& pd) {
    const bool inq = a.flags & APS_INPUT_QUANTIZED;
    const bool outs = a.flags & APS_OUTPUT_SCALED;
    int F[4], Fo[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        F[e] = (inq ? 0 : ft[e]) + f.k;
        Fo[e] = -((outs ? 0 : ft[e]) + f.k);
    }
    bool bad[4] = {false, false, false, false};
    float S[4], cS[4], T[4], cT[4];
    const float* p = a.G + j;
    const int64_t ld = a.ld;
    const int k = 1 << od.log2k;
    int r = 1;  // index of the next add in the order
    stream_rows(
        a.W, [&](int rr) { return ld4(p + (int64_t)order_row(rr, seg, od) * ld); }, [&]() { flush_out(a, pd); },
        [&](const f4& x) {
            const float xs[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                S[e] = quant<V>(xs[e], F[e], f, bad[e]);  // master of the first group
                cS[e] = 0.0f;
                T[e] = 0.0f;
                cT[e] = 0.0f;
            }
        },
        [&](const f4& x, bool valid) {
            if (valid) {
                const float xs[4] = {x.x, x.y, x.z, x.w};
                if ((r & (k - 1)) == 0) {
                    // a new group starts: fold the finished group sum into the ring
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        if (r == k) {
                            T[e] = S[e];
                        } else {
                            chain_step<V, KAHAN>(T[e], cT[e], S[e], f, bad[e]);
                        }
                        S[e] = quant<V>(xs[e], F[e], f, bad[e]);
                        cS[e] = 0.0f;
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) chain_step<V, KAHAN>(S[e], cS[e], quant<V>(xs[e], F[e], f, bad[e]), f, bad[e]);
                }
            }
            ++r;
        });
    float s[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if (od.ng == 1) {
            s[e] = S[e];
        } else {
            chain_step<V, KAHAN>(T[e], cT[e], S[e], f, bad[e]);
            s[e] = T[e];
        }
        s[e] = finish<V>(s[e], bad[e]);
    }
    pd.o.x = __builtin_amdgcn_ldexpf(s[0], Fo[0]);
    pd.o.y = __builtin_amdgcn_ldexpf(s[1], Fo[1]);
    pd.o.z = __builtin_amdgcn_ldexpf(s[2], Fo[2]);
    pd.o.w = __builtin_amdgcn_ldexpf(s[3], Fo[3]);
    if (a.codes) {
#pragma unroll
        for (int e = 0; e < 4; ++e) pd.c[e] = encode(__builtin_amdgcn_ldexpf(s[e], -f.k), f);
    }
    pd.j = j;
    pd.lim = lim;
    pd.valid = true;
}

__device__ __forceinline__ int64_t ring_segment(int64_t j, int64_t n, int ng) { return j * ng / n; }

template <int V, bool KAHAN>
__global__ __launch_bounds__(BLOCK) void k_sim_reduce_ex(ReduceArgs a, Layers ly, Pal pal, Order od) {
    const int64_t nchunks = (ly.n + CH - 1) / CH;
    int64_t cb, ce;
    block_range(nchunks, cb, ce);
    int hint = 0;
    PendingOut pd;
    pd.valid = false;
    for (int64_t c = cb; c < ce; ++c) {
        const int64_t start = c * CH;
        const int64_t end = min(start + CH, ly.n);
        const ChunkInfo ci = chunk_layers(ly, start, end, hint);
        hint = ci.i0;
        const int64_t seg = ring_segment(start, ly.n, od.ng);
        if (ci.mixed || seg != ring_segment(end - 1, ly.n, od.ng)) continue;  // k_sim_reduce_ex_slow
        const FmtK& f = pal.f[ci.pidx];
        if (f.variant != V) continue;
        const int64_t j = start + (int64_t)threadIdx.x * VEC;
        if (j >= end) continue;
        int32_t ft[4];
        if (ci.i0 == ci.i1) {
            const int32_t t = ly.scale_exp ? clamp_exp(cld(ly.scale_exp, ci.i0)) : 0;
            ft[0] = ft[1] = ft[2] = ft[3] = t;
        } else {
            elem_scales(ly, ci, j, ft);
        }
        reduce_vec_ex<V, KAHAN>(a, f, j, end, ft, (int)seg, od, pd);
    }
    flush_out(a, pd);
}

// One element through the whole ordered chain, any variant.
template <int V, bool KAHAN>
__device__ float reduce_elem_ex(const ReduceArgs& a, const FmtK& f, int64_t j, int F, int seg, const Order& od) {
    bool bad = false;
    const int k = 1 << od.log2k;
    auto q = [&](int r) { return quant<V>(a.G[(int64_t)order_row(r, seg, od) * a.ld + j], F, f, bad); };
    float T = 0.0f, cT = 0.0f;
    for (int gi = 0; gi < od.ng; ++gi) {
        float S = q(gi * k), cS = 0.0f;
        for (int m = 1; m < k; ++m) chain_step<V, KAHAN>(S, cS, q(gi * k + m), f, bad);
        if (gi == 0)
            T = S;
        else
            chain_step<V, KAHAN>(T, cT, S, f, bad);
    }
    return finish<V>(T, bad);
}

template <bool KAHAN>
__device__ float reduce_elem_ex_any(const ReduceArgs& a, const FmtK& f, int64_t j, int F, int seg, const Order& od) {
    switch (f.variant) {
        case V_INT_F32: return reduce_elem_ex<V_INT_F32, KAHAN>(a, f, j, F, seg, od);
        case V_INT_F64: return reduce_elem_ex<V_INT_F64, KAHAN>(a, f, j, F, seg, od);
        case V_INT_EXACT: return reduce_elem_ex<V_INT_EXACT, KAHAN>(a, f, j, F, seg, od);
        case V_INT_M0: return reduce_elem_ex<V_INT_M0, KAHAN>(a, f, j, F, seg, od);
        case V_TOP_F32: return reduce_elem_ex<V_TOP_F32, KAHAN>(a, f, j, F, seg, od);
        case V_TOP_F64: return reduce_elem_ex<V_TOP_F64, KAHAN>(a, f, j, F, seg, od);
        case V_TOP_M0: return reduce_elem_ex<V_TOP_M0, KAHAN>(a, f, j, F, seg, od);
        case V_LOW_F32: return reduce_elem_ex<V_LOW_F32, KAHAN>(a, f, j, F, seg, od);
        case V_LOW_F64: return reduce_elem_ex<V_LOW_F64, KAHAN>(a, f, j, F, seg, od);
        default: return reduce_elem_ex<V_LOW_M0, KAHAN>(a, f, j, F, seg, od);
    }
}

// Chunks that mix palette entries or cross a ring-segment boundary, one block
// per chunk (blocks of other chunks return at once); element pairs per
// thread so that a byte of nibble codes has one writer.
template <bool KAHAN>
__global__ __launch_bounds__(BLOCK) void k_sim_reduce_ex_slow(ReduceArgs a, Layers ly, Pal pal, Order od) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    const int64_t start = (int64_t)blockIdx.x * CH;
    if (start >= ly.n) return;
    const int64_t end = min(start + CH, ly.n);
    const ChunkInfo ci = chunk_layers(ly, start, end, 0);
    if (!ci.mixed && ring_segment(start, ly.n, od.ng) == ring_segment(end - 1, ly.n, od.ng)) return;
    for (int64_t j0 = start + 2 * (int64_t)threadIdx.x; j0 < end; j0 += 2 * BLOCK) {
        uint32_t cd[2] = {0, 0};
        for (int e = 0; e < 2; ++e) {
            const int64_t j = j0 + e;
            if (j >= end) break;
            const int li = find_layer(ly.offsets, ly.L, j, 0);
            const FmtK& f = spal[ly.fmt_idx ? ly.fmt_idx[li] : 0];
            const int32_t ft = ly.scale_exp ? clamp_exp(ly.scale_exp[li]) : 0;
            const int F = ((a.flags & APS_INPUT_QUANTIZED) ? 0 : ft) + f.k;
            const int Fo = -(((a.flags & APS_OUTPUT_SCALED) ? 0 : ft) + f.k);
            const float sv = reduce_elem_ex_any<KAHAN>(a, f, j, F, (int)ring_segment(j, ly.n, od.ng), od);
            if (a.out) a.out[j] = __builtin_amdgcn_ldexpf(sv, Fo);
            cd[e] = encode(__builtin_amdgcn_ldexpf(sv, -f.k), f);
            if (a.codes && a.code_cls != 0) put_code(a.codes, j, cd[e], a.code_cls);
        }
        if (a.codes && a.code_cls == 0) {
            uint8_t* q = a.codes + (j0 >> 1);
            *q = (j0 + 1 < end) ? (uint8_t)((cd[0] & 15u) | ((cd[1] & 15u) << 4))
                                : (uint8_t)((*q & 0xF0u) | (cd[0] & 15u));
        }
    }
}

// ================================================ K4c: reduce of packed codes

struct CodesArgs {
    const uint8_t* __restrict__ codes;  // W rows of packed codes
    float* __restrict__ out;
    uint8_t* __restrict__ codes_out;
    int64_t row_bytes;  // bytes per code row (a multiple of 16)
    int32_t W;
    uint32_t flags;
};

// Per-element scale exponents for N consecutive elements from j.
template <int N>
__device__ __forceinline__ void elem_scales_n(const Layers& ly, const ChunkInfo& ci, int64_t j, int32_t* ft) {
    int li = ci.i0;
#pragma unroll
    for (int e = 0; e < N; ++e) {
        while (li < ci.i1 && ly.offsets[li + 1] <= j + e) ++li;
        ft[e] = ly.scale_exp ? clamp_exp(ly.scale_exp[li]) : 0;
    }
}

// Code e (0..EPT-1) of a thread's 16-byte slice.
template <int CC>
__device__ __forceinline__ uint32_t slice_code(const f4& v, int e) {
    const uint32_t w[4] = {f2u(v.x), f2u(v.y), f2u(v.z), f2u(v.w)};
    if constexpr (CC == 0) return (w[e >> 3] >> ((e & 7) * 4)) & 15u;
    else if constexpr (CC == 1) return (w[e >> 2] >> ((e & 3) * 8)) & 255u;
    else return (w[e >> 1] >> ((e & 1) * 16)) & 0xFFFFu;
}

// The W-worker rounded sum of already scaled and cast gradients given as
// packed codes (the low-precision values the workers exchange).  A thread
// owns the codes in 16 bytes of each row: 32 nibble, 16 byte or 8 uint16
// codes.  Codes of up to 8 bits decode through a table of working-domain
// values in LDS; 16-bit codes decode arithmetically.
template <int V, int CC>
__global__ __launch_bounds__(BLOCK) void k_sim_reduce_codes(CodesArgs a, Layers ly, Pal pal) {
    constexpr int EPT = CC == 0 ? 32 : (CC == 1 ? 16 : 8);
    constexpr int64_t CHC = (int64_t)BLOCK * EPT;
    __shared__ float lut[256];
    int lut_pidx = -1;
    const int64_t nchunks = (ly.n + CHC - 1) / CHC;
    int64_t cb, ce;
    block_range(nchunks, cb, ce);
    int hint = 0;
    for (int64_t c = cb; c < ce; ++c) {
        const int64_t start = c * CHC;
        const int64_t end = min(start + CHC, ly.n);
        const ChunkInfo ci = chunk_layers(ly, start, end, hint);
        hint = ci.i0;
        if (ci.mixed) continue;
        const FmtK& f = pal.f[ci.pidx];
        if (f.variant != V) continue;
        if constexpr (CC < 2) {
            if (ci.pidx != lut_pidx) {  // uniform
                __syncthreads();
                for (int t = threadIdx.x; t < (CC == 0 ? 16 : 256); t += BLOCK)
                    lut[t] = __builtin_amdgcn_ldexpf(decode((uint32_t)t, f), f.k);
                __syncthreads();
                lut_pidx = ci.pidx;
            }
        }
        const int64_t j = start + (int64_t)threadIdx.x * EPT;
        if (j >= end) continue;
        const uint8_t* p = a.codes + code_byte(j, CC);
        const int64_t rb = a.row_bytes;
        float s[EPT];
        uint32_t bad = 0;
        auto dec = [&](uint32_t code) -> float {
            if constexpr (CC < 2) return lut[code];
            else return __builtin_amdgcn_ldexpf(decode(code, f), f.k);
        };
        stream_rows(
            a.W, [&](int r) { return ld4((const float*)(p + (int64_t)r * rb)); }, [&]() {},
            [&](const f4& v) {
#pragma unroll
                for (int e = 0; e < EPT; ++e) s[e] = dec(slice_code<CC>(v, e));
            },
            [&](const f4& v, bool valid) {
                if (valid) {
                    // all of the row's table reads first, so their latencies
                    // overlap instead of each add waiting for its own read
                    float d[EPT];
#pragma unroll
                    for (int e = 0; e < EPT; ++e) d[e] = dec(slice_code<CC>(v, e));
                    if constexpr (CC < 2) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int e = 0; e < EPT; ++e) {
                        bool b = false;
                        s[e] = accum<V>(s[e], d[e], f, b);
                        if constexpr (VT<V>::m0) bad |= (uint32_t)b << e;
                    }
                }
            });
        // output exponents, per element when the chunk crosses layers
        const int32_t fdom = ((a.flags & APS_OUTPUT_SCALED) ? 0 : 1);
        int32_t ft[EPT];
        if (ci.i0 == ci.i1) {
            const int32_t t = ly.scale_exp ? clamp_exp(cld(ly.scale_exp, ci.i0)) : 0;
#pragma unroll
            for (int e = 0; e < EPT; ++e) ft[e] = t;
        } else {
            elem_scales_n<EPT>(ly, ci, j, ft);
        }
        float o[EPT];
        uint32_t cw[4] = {0, 0, 0, 0};
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
            const float se = VT<V>::m0 ? (((bad >> e) & 1u) ? __builtin_nanf("") : s[e]) : s[e];
            o[e] = __builtin_amdgcn_ldexpf(se, -(fdom * ft[e] + f.k));
            if (a.codes_out) {
                const uint32_t cd = encode(__builtin_amdgcn_ldexpf(se, -f.k), f);
                if constexpr (CC == 0) cw[e >> 3] |= (cd & 15u) << ((e & 7) * 4);
                else if constexpr (CC == 1) cw[e >> 2] |= (cd & 255u) << ((e & 3) * 8);
                else cw[e >> 1] |= (cd & 0xFFFFu) << ((e & 1) * 16);
            }
        }
        if (j + EPT <= end) {
            if (a.out) {
#pragma unroll
                for (int q = 0; q < EPT / 4; ++q) {
                    const f4 v = {o[4 * q], o[4 * q + 1], o[4 * q + 2], o[4 * q + 3]};
                    __builtin_nontemporal_store(v, (f4*)(a.out + j + 4 * q));
                }
            }
            if (a.codes_out) {
                const u4v v = {cw[0], cw[1], cw[2], cw[3]};
                __builtin_nontemporal_store(v, (u4v*)(a.codes_out + code_byte(j, CC)));
            }
        } else {
            // ragged end of the gradient: element by element
            for (int e = 0; e < EPT && j + e < end; ++e) {
                if (a.out) a.out[j + e] = o[e];
                if (a.codes_out) {
                    const int64_t jj = j + e;
                    if constexpr (CC == 0) {
                        const uint32_t cd = (cw[e >> 3] >> ((e & 7) * 4)) & 15u;
                        uint8_t* pb = a.codes_out + (jj >> 1);
                        const int sh = (int)(jj & 1) * 4;
                        *pb = (uint8_t)((*pb & ~(15u << sh)) | (cd << sh));
                    } else if constexpr (CC == 1) {
                        a.codes_out[jj] = (uint8_t)(cw[e >> 2] >> ((e & 3) * 8));
                    } else {
                        *(uint16_t*)(a.codes_out + 2 * jj) = (uint16_t)(cw[e >> 1] >> ((e & 1) * 16));
                    }
                }
            }
        }
    }
}

// Mixed-format chunks of the codes reduce: element pairs per thread, any variant.
template <int V>
__device__ float reduce_codes_elem(const CodesArgs& a, const FmtK& f, int cc, int64_t j) {
    bool bad = false;
    const int64_t cb = code_byte(j, cc);
    auto get = [&](int w) -> float {
        const uint8_t* row = a.codes + (int64_t)w * a.row_bytes;
        uint32_t code;
        if (cc == 0)
            code = (row[cb] >> ((j & 1) * 4)) & 15u;
        else if (cc == 1)
            code = row[cb];
        else
            code = *(const uint16_t*)(row + cb);
        return __builtin_amdgcn_ldexpf(decode(code, f), f.k);
    };
    float s = get(0);
    for (int w = 1; w < a.W; ++w) s = accum<V>(s, get(w), f, bad);
    return finish<V>(s, bad);
}

__device__ float reduce_codes_any(const CodesArgs& a, const FmtK& f, int cc, int64_t j) {
    switch (f.variant) {
        case V_INT_F32: return reduce_codes_elem<V_INT_F32>(a, f, cc, j);
        case V_INT_F64: return reduce_codes_elem<V_INT_F64>(a, f, cc, j);
        case V_INT_EXACT: return reduce_codes_elem<V_INT_EXACT>(a, f, cc, j);
        case V_INT_M0: return reduce_codes_elem<V_INT_M0>(a, f, cc, j);
        case V_TOP_F32: return reduce_codes_elem<V_TOP_F32>(a, f, cc, j);
        case V_TOP_F64: return reduce_codes_elem<V_TOP_F64>(a, f, cc, j);
        case V_TOP_M0: return reduce_codes_elem<V_TOP_M0>(a, f, cc, j);
        case V_LOW_F32: return reduce_codes_elem<V_LOW_F32>(a, f, cc, j);
        case V_LOW_F64: return reduce_codes_elem<V_LOW_F64>(a, f, cc, j);
        default: return reduce_codes_elem<V_LOW_M0>(a, f, cc, j);
    }
}

// One block per layer boundary; the chunk (of the codes reduce's chunk size)
// owning the first boundary strictly inside it, when it mixes palette entries.
template <int CC>
__global__ __launch_bounds__(BLOCK) void k_sim_reduce_codes_mixed(CodesArgs a, Layers ly, Pal pal) {
    constexpr int64_t CHC = (int64_t)BLOCK * (CC == 0 ? 32 : (CC == 1 ? 16 : 8));
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    const int b = blockIdx.x;
    if (b < 1 || b >= ly.L) return;
    const int64_t pb = cld(ly.offsets, b);
    if (pb <= 0 || pb >= ly.n || pb % CHC == 0) return;
    const int64_t start = pb / CHC * CHC;
    const int64_t end = min(start + CHC, ly.n);
    if (cld(ly.offsets, b - 1) > start) return;
    if (!chunk_layers(ly, start, end, 0).mixed) return;
    for (int64_t j0 = start + 2 * (int64_t)threadIdx.x; j0 < end; j0 += 2 * BLOCK) {
        uint32_t cd[2] = {0, 0};
        for (int e = 0; e < 2; ++e) {
            const int64_t j = j0 + e;
            if (j >= end) break;
            const int li = find_layer(ly.offsets, ly.L, j, 0);
            const FmtK& f = spal[ly.fmt_idx[li]];
            const int32_t ft = ly.scale_exp ? clamp_exp(ly.scale_exp[li]) : 0;
            const float sv = reduce_codes_any(a, f, CC, j);
            const int fd = (a.flags & APS_OUTPUT_SCALED) ? 0 : ft;
            if (a.out) a.out[j] = __builtin_amdgcn_ldexpf(sv, -(fd + f.k));
            cd[e] = encode(__builtin_amdgcn_ldexpf(sv, -f.k), f);
            if (a.codes_out && CC != 0) put_code(a.codes_out, j, cd[e], CC);
        }
        if (a.codes_out && CC == 0) {
            uint8_t* q = a.codes_out + (j0 >> 1);
            *q = (j0 + 1 < end) ? (uint8_t)((cd[0] & 15u) | ((cd[1] & 15u) << 4))
                                : (uint8_t)((*q & 0xF0u) | (cd[0] & 15u));
        }
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

__device__ float reduce_elem_any(const ReduceArgs& a, const FmtK& f, int64_t j, int F) {
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

// Each thread owns an element pair (2t, 2t+1) of the chunk, so a byte of
// nibble codes is written by one thread only.
__global__ __launch_bounds__(BLOCK) void k_sim_reduce_mixed(ReduceArgs a, Layers ly, Pal pal) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    int64_t start, end;
    if (!mixed_chunk_of_boundary(ly, blockIdx.x, start, end)) return;
    for (int64_t j0 = start + 2 * (int64_t)threadIdx.x; j0 < end; j0 += 2 * BLOCK) {
        uint32_t c[2] = {0, 0};
        for (int e = 0; e < 2; ++e) {
            const int64_t j = j0 + e;
            if (j >= end) break;
            const int li = find_layer(ly.offsets, ly.L, j, 0);
            const FmtK& f = spal[ly.fmt_idx[li]];
            const int32_t ft = ly.scale_exp ? clamp_exp(ly.scale_exp[li]) : 0;
            const int F = ((a.flags & APS_INPUT_QUANTIZED) ? 0 : ft) + f.k;
            const int Fo = -(((a.flags & APS_OUTPUT_SCALED) ? 0 : ft) + f.k);
            const float s = reduce_elem_any(a, f, j, F);
            if (a.out) a.out[j] = __builtin_amdgcn_ldexpf(s, Fo);
            c[e] = encode(__builtin_amdgcn_ldexpf(s, -f.k), f);
            if (a.codes && a.code_cls != 0) put_code(a.codes, j, c[e], a.code_cls);
        }
        if (a.codes && a.code_cls == 0) {
            uint8_t* pb = a.codes + (j0 >> 1);
            *pb = (j0 + 1 < end) ? (uint8_t)((c[0] & 15u) | ((c[1] & 15u) << 4))
                                 : (uint8_t)((*pb & 0xF0u) | (c[0] & 15u));
        }
    }
}

// ============================================ K5: one-pass synchronisation
//
// A layer's scale 2^ft is known only after the max over every worker and
// element of the layer, which would make the fused sum a second full read
// of the W rows.  It need not be.  Power-of-two scaling commutes with
// rounding to m+1 significant bits (Sec. 3.3.1); only the format's
// subnormal range and its overflow depend on ft.  So the first pass sums
// the UNSCALED values, rounding to m+1 significant bits with an unbounded
// exponent (rho below), while it takes the max.  Once the scales are known,
// its result is the exact result of the scaled path for every element in
// which each nonzero input x_k satisfies |x_k| >= T = max(2^(emin - ft),
// 2^-126), or arrives (k >= 1) when the unscaled partial sum has
// |s_(k-1)| >= 2^(m+3) * T, in a layer with 0 < N * ghat <= 2^127 (or an
// all-zero layer), when N = W is a power of two:
//   * an x with |x| >= T is an fp32 normal, x * 2^ft is exact and in the
//     format's normal range, so R(x * 2^ft) = 2^ft * rho(x);
//   * a smaller x casts to at most T * 2^ft scaled (T unscaled), at most a
//     quarter of the partial sum's smallest gap once |s| >= 2^(m+3) * T,
//     so both chains leave the sum unchanged;
//   * partial sums are then multiples of 2^(emin - ft - m): a sum below
//     2^(emin - ft) is exact both ways, one above rounds the same way both
//     ways (fp32 add + rho = rho of the exact sum for m <= 10);
//   * nothing overflows: every |q| <= 2^emax / N, and the worst chain, all
//     q equal to that bound, counts exactly up to min(N, 2^(m+1)) of them
//     and then stays (ties to even; m = 0: 1, 2, 4, 4, ...), so every
//     partial sum stays at or below 2^emax; unscaled, at or below 2^127.
// The first pass keeps per element one byte: the exponent field of
// min_k max(|x_k|, |s_(k-1)| * 2^-(m+3)) over the nonzero x_k (the first
// term alone), less one ulp; it lies below T's exponent whenever the test
// fails.  The second pass lists the chunks holding such an element (from
// one byte per 256 elements), then recomputes those elements through the
// scaled path: one wave per element when few elements of a chunk fail, the
// whole chunk with the streaming kernel's row walk when many do.

// rho: round an fp32 bit pattern to m+1 significant bits, ties to the even
// significand (m = 0: up, the even multiple of the quantum), exponent
// unbounded.  lw is the width of the tie bit (1, or 0 when m = 0).
__device__ __forceinline__ uint32_t rho(uint32_t b, uint32_t half, uint32_t sh, uint32_t lw, uint32_t mask) {
    return (b + half + __builtin_amdgcn_ubfe(b, sh, lw)) & mask;
}

// Device view of the caller's workspace (layout in sync_layout()).
struct SyncWs {
    uint8_t* __restrict__ minb;  // [round_up(n, CH)] per-element exponent byte
    uint8_t* __restrict__ wmin;  // [4 per chunk] min of minb over each wave's 256 elements
    int32_t* __restrict__ thr;   // [L] repair threshold per layer
    uint32_t* __restrict__ count;  // chunks listed for repair
    int32_t* __restrict__ list;    // [nchunks] those chunks
};

struct SyncArgs {
    const float* __restrict__ G;
    float* __restrict__ out;
    int64_t ld;
    int32_t W;
};

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
    for (int o = 32; o > 0; o >>= 1) v = min(v, (uint32_t)__shfl_xor((int)v, o, 64));
    return v;
}

// A thread's finished first-pass results for 4 elements, stored after the
// next chunk's loads have been issued (see PendingOut); lane 0 of a wave also
// holds the wave's minimum byte.
struct PendingSync {
    f4 o;
    uint32_t mb;  // the 4 exponent bytes, element j in the low byte
    uint32_t wb;  // wave minimum (lane 0)
    int64_t j, lim, c;
    bool valid;
};

__device__ __forceinline__ void flush_sync(const SyncArgs& a, const SyncWs& ws, PendingSync& pd) {
    if (!pd.valid) return;
    pd.valid = false;
    const int64_t j = pd.j, lim = pd.lim;
    if (j + 4 <= lim) {
        __builtin_nontemporal_store(pd.o, (f4*)(a.out + j));
    } else {
        if (j < lim) a.out[j] = pd.o.x;
        if (j + 1 < lim) a.out[j + 1] = pd.o.y;
        if (j + 2 < lim) a.out[j + 2] = pd.o.z;
    }
    // the byte array is padded to whole chunks: a full word is always in bounds
    __builtin_nontemporal_store(pd.mb, (uint32_t*)(ws.minb + j));
    if ((threadIdx.x & 63) == 0) ws.wmin[pd.c * 4 + (threadIdx.x >> 6)] = (uint8_t)pd.wb;
}

__global__ __launch_bounds__(BLOCK) void k_sync_spec(SyncArgs a, SyncWs ws, Layers ly, Pal pal,
                                                    uint32_t* __restrict__ maxabs) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    __shared__ uint32_t red[BLOCK / 64];
    pal_to_lds(pal, spal);
    const int64_t nchunks = (ly.n + CH - 1) / CH;
    int64_t cb, ce;
    block_range(nchunks, cb, ce);
    int hint = 0;
    uint32_t run = 0;  // running max of layer run_layer (chunks inside one layer)
    int run_layer = -1;
    PendingSync pd;
    pd.valid = false;
    const f4 neg0 = {-0.0f, -0.0f, -0.0f, -0.0f};
    for (int64_t c = cb; c < ce; ++c) {
        const int64_t start = c * CH;
        const int64_t end = min(start + CH, ly.n);
        const ChunkInfo ci = chunk_layers(ly, start, end, hint);
        hint = ci.i0;
        const int64_t j = start + (int64_t)threadIdx.x * VEC;
        uint32_t mx0 = 0, mx1 = 0, mx2 = 0, mx3 = 0;
        uint32_t tmin = 255u;  // this thread's smallest exponent byte
        if (j < end) {
            uint32_t hf[4], sh[4], lw[4], mk[4];
            float sc[4];  // 2^-(m+3)
            if (!ci.mixed) {
                const FmtK& f = pal.f[ci.pidx];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    hf[e] = f.half;
                    sh[e] = f.sh;
                    lw[e] = f.lsbw;
                    mk[e] = f.mask;
                    sc[e] = u2f((uint32_t)(124 - f.m) << 23);
                }
            } else {
                int li = ci.i0;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    while (li < ci.i1 && ly.offsets[li + 1] <= j + e) ++li;
                    const FmtK& f = spal[ly.fmt_idx[li]];
                    hf[e] = f.half;
                    sh[e] = f.sh;
                    lw[e] = f.lsbw;
                    mk[e] = f.mask;
                    sc[e] = u2f((uint32_t)(124 - f.m) << 23);
                }
            }
            uint32_t mn0, mn1, mn2, mn3;
            float s0, s1, s2, s3;
            const float* p = a.G + j;
            const int64_t ld = a.ld;
            stream_rows(
                a.W, [&](int r) { return ld4(p + (int64_t)r * ld); },
                [&]() { flush_sync(a, ws, pd); },
                [&](const f4& x) {
                    const uint32_t b0 = f2u(x.x), b1 = f2u(x.y), b2 = f2u(x.z), b3 = f2u(x.w);
                    mx0 = b0 & 0x7FFFFFFFu;
                    mx1 = b1 & 0x7FFFFFFFu;
                    mx2 = b2 & 0x7FFFFFFFu;
                    mx3 = b3 & 0x7FFFFFFFu;
                    mn0 = mx0 - 1u;  // a zero wraps to the top and never wins the min
                    mn1 = mx1 - 1u;
                    mn2 = mx2 - 1u;
                    mn3 = mx3 - 1u;
                    s0 = u2f(rho(b0, hf[0], sh[0], lw[0], mk[0]));
                    s1 = u2f(rho(b1, hf[1], sh[1], lw[1], mk[1]));
                    s2 = u2f(rho(b2, hf[2], sh[2], lw[2], mk[2]));
                    s3 = u2f(rho(b3, hf[3], sh[3], lw[3], mk[3]));
                },
                [&](const f4& r, bool valid) {
                    // a row past the last one counts as -0: no change to any of the four
                    const f4 v = valid ? r : neg0;
                    const uint32_t b0 = f2u(v.x), b1 = f2u(v.y), b2 = f2u(v.z), b3 = f2u(v.w);
                    const uint32_t a0 = b0 & 0x7FFFFFFFu, a1 = b1 & 0x7FFFFFFFu;
                    const uint32_t a2 = b2 & 0x7FFFFFFFu, a3 = b3 & 0x7FFFFFFFu;
                    mx0 = max(mx0, a0);
                    mx1 = max(mx1, a1);
                    mx2 = max(mx2, a2);
                    mx3 = max(mx3, a3);
                    // the term's magnitude, or the sum it meets scaled down by 2^(m+3)
                    mn0 = min(mn0, max(a0 - 1u, f2u(u2f(f2u(s0) & 0x7FFFFFFFu) * sc[0])));
                    mn1 = min(mn1, max(a1 - 1u, f2u(u2f(f2u(s1) & 0x7FFFFFFFu) * sc[1])));
                    mn2 = min(mn2, max(a2 - 1u, f2u(u2f(f2u(s2) & 0x7FFFFFFFu) * sc[2])));
                    mn3 = min(mn3, max(a3 - 1u, f2u(u2f(f2u(s3) & 0x7FFFFFFFu) * sc[3])));
                    s0 = u2f(rho(f2u(s0 + u2f(rho(b0, hf[0], sh[0], lw[0], mk[0]))), hf[0], sh[0], lw[0], mk[0]));
                    s1 = u2f(rho(f2u(s1 + u2f(rho(b1, hf[1], sh[1], lw[1], mk[1]))), hf[1], sh[1], lw[1], mk[1]));
                    s2 = u2f(rho(f2u(s2 + u2f(rho(b2, hf[2], sh[2], lw[2], mk[2]))), hf[2], sh[2], lw[2], mk[2]));
                    s3 = u2f(rho(f2u(s3 + u2f(rho(b3, hf[3], sh[3], lw[3], mk[3]))), hf[3], sh[3], lw[3], mk[3]));
                });
            const uint32_t e0 = min(mn0 >> 23, 255u), e1 = min(mn1 >> 23, 255u);
            const uint32_t e2 = min(mn2 >> 23, 255u), e3 = min(mn3 >> 23, 255u);
            pd.o.x = s0;
            pd.o.y = s1;
            pd.o.z = s2;
            pd.o.w = s3;
            pd.mb = e0 | (e1 << 8) | (e2 << 16) | (e3 << 24);
            pd.j = j;
            pd.lim = end;
            pd.c = c;
            pd.valid = true;
            // elements past the end of the gradient (row padding) do not count
            tmin = e0;
            if (j + 1 < end) tmin = min(tmin, e1); else mx1 = 0;
            if (j + 2 < end) tmin = min(tmin, e2); else mx2 = 0;
            if (j + 3 < end) tmin = min(tmin, e3); else mx3 = 0;
        }
        // every lane of the wave takes part; lane 0 has the wave's first
        // element, so its pending record exists whenever the wave has one
        pd.wb = wave_min_u32(tmin);
        if (ci.i0 == ci.i1) {
            const uint32_t v = max(max(mx0, mx1), max(mx2, mx3));
            if (ci.i0 != run_layer) {
                if (run_layer >= 0) block_max_atomic(run, maxabs + run_layer, red);
                run_layer = ci.i0;
                run = 0;
            }
            run = max(run, v);
        } else {
            const uint32_t mv[4] = {mx0, mx1, mx2, mx3};
            for (int li = ci.i0; li <= ci.i1; ++li) {
                const int64_t lo = cld(ly.offsets, li), hi = cld(ly.offsets, li + 1);
                uint32_t v = 0;
                if (j < end)
                    for (int e = 0; e < 4; ++e)
                        if (j + e >= lo && j + e < hi) v = max(v, mv[e]);
                block_max_atomic(v, maxabs + li, red);
            }
        }
    }
    if (run_layer >= 0) block_max_atomic(run, maxabs + run_layer, red);
    flush_sync(a, ws, pd);
}

// Scale exponents (as k_scales) and the per-layer repair threshold: an
// element is recomputed when its exponent byte is below thr[i].  thr = 256
// recomputes the whole layer (ghat INF/NaN, N * ghat = INF or above 2^127);
// an all-zero layer needs nothing.  Also clears the repair list.
__global__ void k_sync_layers(const uint32_t* __restrict__ maxabs, int32_t L, int32_t N, Pal pal,
                              const uint8_t* __restrict__ fmt_idx, int32_t* __restrict__ scale_exp, SyncWs ws) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0) *ws.count = 0u;
    if (i >= L) return;
    const FmtK& f = spal[fmt_idx ? fmt_idx[i] : 0];
    const uint32_t gb = maxabs[i] & 0x7FFFFFFFu;
    int32_t r = 0, th = 256;
    if (gb == 0) {
        th = 0;
    } else if (gb < 0x7F800000u) {
        const float t = (float)N * u2f(gb);
        const uint32_t tb = f2u(t);
        if (tb < 0x7F800000u) {
            const int cl = ceil_log2_bits(tb);
            r = f.emax - cl;
            // smallest safe nonzero magnitude: 2^max(emin - ft, -126), as an exponent field
            if (cl <= 127) th = max(f.emin - r + 127, 1);
        }
    }
    scale_exp[i] = r;
    ws.thr[i] = th;
}

// Largest i in [0, L-1] with offsets[i] <= pos, for pos < n (per lane).
__device__ __forceinline__ int layer_of(const int64_t* __restrict__ off, int L, int64_t pos) {
    int lo = 0, hi = L;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (off[mid] <= pos) lo = mid; else hi = mid;
    }
    return lo;
}

// One thread per chunk: list the chunks (single palette entry) holding an
// element whose byte is below its layer's threshold.  The test is on the
// chunk's minimum byte against the largest threshold among its layers, so
// it never misses one; the repair looks at each element.
__global__ void k_sync_scan(Layers ly, SyncWs ws) {
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t nchunks = (ly.n + CH - 1) / CH;
    if (c >= nchunks) return;
    const int64_t start = c * CH;
    const int64_t end = min(start + CH, ly.n);
    const uint32_t w4 = *(const uint32_t*)(ws.wmin + 4 * c);
    uint32_t cm = 255u;
    for (int wv = 0; wv < 4; ++wv)
        if (start + 256 * wv < end) cm = min(cm, (w4 >> (8 * wv)) & 0xFFu);
    const int i0 = layer_of(ly.offsets, ly.L, start), i1 = layer_of(ly.offsets, ly.L, end - 1);
    int32_t th = 0;
    bool mixed = false;
    const int p0 = ly.fmt_idx ? ly.fmt_idx[i0] : 0;
    for (int i = i0; i <= i1; ++i) {
        if (ly.offsets[i] == ly.offsets[i + 1]) continue;  // empty layer
        th = max(th, ws.thr[i]);
        if (ly.fmt_idx && ly.fmt_idx[i] != p0) mixed = true;
    }
    if (!mixed && (int32_t)cm < th) ws.list[atomicAdd(ws.count, 1u)] = (int32_t)c;
}

constexpr int SPARSE_MAX = 16;  // flagged elements per chunk repaired one wave each

// The exact scaled path for one element, run by a whole wave: each lane
// loads and casts a different worker's value, then every lane walks the
// casts in worker order (one readlane per add) and lane 0 stores.
template <int V>
__device__ void repair_one(const ReduceArgs& a, const FmtK& f, int64_t j, int F) {
    const int lane = threadIdx.x & 63;
    const float* p = a.G + j;
    bool badl = false, bads = false;
    float s = 0.0f;
    for (int base = 0; base < a.W; base += 256) {
        float q[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int r = base + 64 * u + lane;
            q[u] = quant<V>(r < a.W ? p[(int64_t)r * a.ld] : -0.0f, F, f, badl);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int r0 = base + 64 * u;
            const int cnt = min(64, a.W - r0);
            for (int t = 0; t < cnt; ++t) {
                const float qt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(q[u]), t));
                if (r0 + t == 0)
                    s = qt;
                else
                    s = accum<V>(s, qt, f, bads);
            }
        }
    }
    const bool bad = bads || (__ballot(badl) != 0);
    s = finish<V>(s, bad);
    if (lane == 0) a.out[j] = __builtin_amdgcn_ldexpf(s, -F);
}

// Second pass over the listed chunks of one variant's format, one wave per
// chunk: find the flagged elements (16 bytes per lane), then repair them one
// after another (at most SPARSE_MAX), or rerun the whole chunk through the
// streaming row walk, a quarter at a time.  Waves stride over the list; its
// length is read on the device.
template <int V>
__global__ __launch_bounds__(BLOCK) void k_sync_repair(ReduceArgs a, Layers ly, Pal pal, SyncWs ws) {
    const uint32_t total = *ws.count;
    const int lane = threadIdx.x & 63;
    const int64_t nw = (int64_t)gridDim.x * (BLOCK / 64);
    for (int64_t k = __builtin_amdgcn_readfirstlane((int)(blockIdx.x * (BLOCK / 64) + (threadIdx.x >> 6))); k < total;
         k += nw) {
        const int64_t start = (int64_t)cld(ws.list, k) * CH;
        const int64_t end = min(start + CH, ly.n);
        const ChunkInfo ci = chunk_layers(ly, start, end, 0);
        const FmtK& f = pal.f[ci.pidx];
        if (f.variant != V) continue;  // another launch owns this format
        // 16 consecutive elements per lane; the byte array is padded to whole chunks
        const int64_t j0 = start + 16 * lane;
        const u4v w = *(const u4v*)(ws.minb + j0);
        uint32_t mask = 0;
        if (ci.i0 == ci.i1) {  // one layer: one threshold, read once
            const int32_t th = cld(ws.thr, ci.i0);
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const uint32_t byte = (w[e >> 2] >> (8 * (e & 3))) & 0xFFu;
                if ((int32_t)byte < th && j0 + e < end) mask |= 1u << e;
            }
        } else {
            int li = ci.i0;
            int64_t next = ly.offsets[li + 1];
            int32_t th = ws.thr[li];
            for (int e = 0; e < 16; ++e) {
                const int64_t jj = j0 + e;
                if (jj >= end) break;
                while (li < ci.i1 && next <= jj) {
                    ++li;
                    next = ly.offsets[li + 1];
                    th = ws.thr[li];
                }
                const uint32_t byte = (w[e >> 2] >> (8 * (e & 3))) & 0xFFu;
                if ((int32_t)byte < th) mask |= 1u << e;
            }
        }
        int cnt = __builtin_popcount(mask);
        for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
        if (cnt > SPARSE_MAX) {
#pragma unroll 1
            for (int qtr = 0; qtr < 4; ++qtr) {
                const int64_t j = start + (int64_t)qtr * 256 + 4 * lane;
                if (j >= end) continue;
                int32_t ft[4];
                if (ci.i0 == ci.i1) {
                    const int32_t t = clamp_exp(cld(ly.scale_exp, ci.i0));
                    ft[0] = ft[1] = ft[2] = ft[3] = t;
                } else {
                    elem_scales(ly, ci, j, ft);
                }
                PendingOut pd;
                pd.valid = false;
                reduce_vec<V>(a, f, j, end, ft, pd);
                flush_out(a, pd);
            }
        } else {
            uint64_t lanes = __ballot(mask != 0);
            while (lanes) {
                const int l = __builtin_ctzll(lanes);
                lanes &= lanes - 1;
                uint32_t m = (uint32_t)__builtin_amdgcn_readlane((int)mask, l);
                while (m) {
                    const int e = __builtin_ctz(m);
                    m &= m - 1;
                    const int64_t jj = start + 16 * l + e;
                    const int lj = find_layer(ly.offsets, ly.L, jj, ci.i0);
                    repair_one<V>(a, f, jj, clamp_exp(cld(ly.scale_exp, lj)) + f.k);
                }
            }
        }
    }
}

// Flagged elements of chunks that mix palette entries, element by element.
__global__ __launch_bounds__(BLOCK) void k_sync_repair_mixed(ReduceArgs a, Layers ly, Pal pal, SyncWs ws) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    int64_t start, end;
    if (!mixed_chunk_of_boundary(ly, blockIdx.x, start, end)) return;
    for (int64_t j = start + threadIdx.x; j < end; j += BLOCK) {
        const int li = find_layer(ly.offsets, ly.L, j, 0);
        if ((int32_t)ws.minb[j] >= ws.thr[li]) continue;
        const FmtK& f = spal[ly.fmt_idx[li]];
        const int F = clamp_exp(ly.scale_exp[li]) + f.k;
        a.out[j] = __builtin_amdgcn_ldexpf(reduce_elem_any(a, f, j, F), -F);
    }
}

// ======================================================= K3: quantize

struct QuantArgs {
    const float* X;
    float* Q;  // may alias X: each element is read before its own store
    uint8_t* __restrict__ codes;
    int64_t ld;
    int32_t W;
    int32_t code_cls;
};

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
template <int V>
__device__ __forceinline__ void quantize_tail(const QuantArgs& a, const FmtK& f, int64_t j, int64_t end,
                                           const int32_t ft[4]) {
#pragma unroll 1
    for (int64_t r = 0; r < a.W; ++r) {
        const int64_t off = r * a.ld + j;
        uint32_t cc[4] = {0, 0, 0, 0};
        for (int e = 0; e < 4 && j + e < end; ++e) {
            const float v = quant_native<V>(a.X[off + e], ft[e] + f.k, f);
            if (a.Q) a.Q[off + e] = v;
            cc[e] = encode(v, f);
        }
        if (a.codes) store_codes4(a.codes + code_byte(r * a.ld, a.code_cls), j, cc, a.code_cls, end);
    }
}

// The cast alone does not depend on the accumulator width, so the F32 and F64
// variants of a class cast alike; the F64 form reads the tie-bit width from the
// format (1 whenever the F32 form applies).
__host__ __device__ constexpr int cast_variant(int v) {
    return v == V_INT_F32 ? V_INT_F64 : (v == V_TOP_F32 ? V_TOP_F64 : (v == V_LOW_F32 ? V_LOW_F64 : v));
}

// What one k_quantize launch writes per row.
enum QuantOut { QO_Q = 0, QO_CODES4 = 1, QO_CODES8 = 2, QO_CODES16 = 3, QO_BOTH = 4 };

// One block walks a range of chunks; for each chunk its threads stream all W
// rows (two register sets of rows in flight), cast each row and store it.
// The stores of a row are fixed at compile time (OUT): a store that is
// conditional inside the streamed loop makes the compiler's load-counter
// waits at the loop's joins far more conservative.
template <int V, int OUT>
__global__ __launch_bounds__(BLOCK) void k_quantize(QuantArgs a, Layers ly, Pal pal) {
    constexpr bool HQ = OUT == QO_Q || OUT == QO_BOTH;
    constexpr bool HC = OUT != QO_Q;
    const int64_t nchunks = (ly.n + CH - 1) / CH;
    int64_t cb, ce;
    block_range(nchunks, cb, ce);
    int hint = 0;
    for (int64_t c = cb; c < ce; ++c) {
        const int64_t start = c * CH;
        const int64_t end = min(start + CH, ly.n);
        const ChunkInfo ci = chunk_layers(ly, start, end, hint);
        hint = ci.i0;
        if (ci.mixed) continue;  // handled by k_quantize_mixed
        const FmtK& f = pal.f[ci.pidx];
        if (cast_variant(f.variant) != V) continue;
        const int64_t j = start + (int64_t)threadIdx.x * VEC;
        if (j >= end) continue;
        int32_t ft[4];
        if (ci.i0 == ci.i1) {
            const int32_t t = ly.scale_exp ? clamp_exp(cld(ly.scale_exp, ci.i0)) : 0;
            ft[0] = ft[1] = ft[2] = ft[3] = t;
        } else {
            elem_scales(ly, ci, j, ft);
        }
        if (j + 4 > end) {
            quantize_tail<V>(a, f, j, end, ft);
            continue;
        }
        const float* p = a.X + j;
        const int64_t ld = a.ld;
        const int cls = OUT == QO_CODES4 ? 0 : (OUT == QO_CODES8 ? 1 : (OUT == QO_CODES16 ? 2 : a.code_cls));
        int64_t r = 0;  // row of the next callback
        auto row = [&](const f4& x, bool valid) {
            if (valid) {
                const f4 v = {quant_native<V>(x.x, ft[0] + f.k, f), quant_native<V>(x.y, ft[1] + f.k, f),
                              quant_native<V>(x.z, ft[2] + f.k, f), quant_native<V>(x.w, ft[3] + f.k, f)};
                if constexpr (HQ) __builtin_nontemporal_store(v, (f4*)(a.Q + j + r * ld));
                if constexpr (HC) {
                    const uint32_t cc[4] = {encode(v.x, f), encode(v.y, f), encode(v.z, f), encode(v.w, f)};
                    store_codes4_full(a.codes + code_byte(r * ld, cls), j, cc, cls);
                }
            }
            ++r;
        };
        stream_rows(
            a.W, [&](int rr) { return ld4(p + (int64_t)rr * ld); }, [&]() {}, [&](const f4& x) { row(x, true); }, row);
    }
}

__device__ float quant_any(float x, int F, const FmtK& f) {
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
        default: return quant_native<V_LOW_M0>(x, F, f);
    }
}

// Mixed-format chunks, all W rows; grid (boundary, worker); element pairs
// per thread as in k_sim_reduce_mixed.
__global__ __launch_bounds__(BLOCK) void k_quantize_mixed(QuantArgs a, Layers ly, Pal pal) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    int64_t start, end;
    if (!mixed_chunk_of_boundary(ly, blockIdx.x, start, end)) return;
    const int64_t w = blockIdx.y;
    uint8_t* row = a.codes ? a.codes + code_byte(w * a.ld, a.code_cls) : nullptr;
    for (int64_t j0 = start + 2 * (int64_t)threadIdx.x; j0 < end; j0 += 2 * BLOCK) {
        uint32_t c[2] = {0, 0};
        for (int e = 0; e < 2; ++e) {
            const int64_t j = j0 + e;
            if (j >= end) break;
            const int li = find_layer(ly.offsets, ly.L, j, 0);
            const FmtK& f = spal[ly.fmt_idx[li]];
            const int32_t ft = ly.scale_exp ? clamp_exp(ly.scale_exp[li]) : 0;
            const int64_t off = w * a.ld + j;
            const float v = quant_any(a.X[off], ft + f.k, f);  // Q may alias X: same element
            if (a.Q) a.Q[off] = v;
            c[e] = encode(v, f);
            if (row && a.code_cls != 0) put_code(row, j, c[e], a.code_cls);
        }
        if (row && a.code_cls == 0) {
            uint8_t* pb = row + (j0 >> 1);
            *pb = (j0 + 1 < end) ? (uint8_t)((c[0] & 15u) | ((c[1] & 15u) << 4))
                                 : (uint8_t)((*pb & 0xF0u) | (c[0] & 15u));
        }
    }
}

// ===================================================== K5: dequantize

struct DeqArgs {
    const float* Q;  // may alias out
    const uint8_t* __restrict__ codes;
    float* out;
    int32_t code_cls;
};

__global__ __launch_bounds__(BLOCK) void k_dequantize(DeqArgs a, Layers ly, Pal pal) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    const int64_t nchunks = (ly.n + CH - 1) / CH;
    int64_t cb, ce;
    block_range(nchunks, cb, ce);
    int hint = 0;
    for (int64_t c = cb; c < ce; ++c) {
        const int64_t start = c * CH;
        const int64_t end = min(start + CH, ly.n);
        const ChunkInfo ci = chunk_layers(ly, start, end, hint);
        hint = ci.i0;
        const int64_t j = start + (int64_t)threadIdx.x * VEC;
        if (j >= end) continue;
        if (ci.i0 == ci.i1 && j + 4 <= end) {
            // one layer: uniform format and exponent, 16-byte accesses
            const FmtK& f = pal.f[ci.pidx];
            const int32_t ft = ly.scale_exp ? clamp_exp(cld(ly.scale_exp, ci.i0)) : 0;
            f4 v;
            if (a.Q) {
                v = *(const f4*)(a.Q + j);
            } else {
                v.x = decode(load_code(a.codes, j, a.code_cls), f);
                v.y = decode(load_code(a.codes, j + 1, a.code_cls), f);
                v.z = decode(load_code(a.codes, j + 2, a.code_cls), f);
                v.w = decode(load_code(a.codes, j + 3, a.code_cls), f);
            }
            const f4 o = {__builtin_amdgcn_ldexpf(v.x, -ft), __builtin_amdgcn_ldexpf(v.y, -ft),
                          __builtin_amdgcn_ldexpf(v.z, -ft), __builtin_amdgcn_ldexpf(v.w, -ft)};
            __builtin_nontemporal_store(o, (f4*)(a.out + j));  // out may alias Q: same elements
            continue;
        }
        int li = ci.i0;
        for (int e = 0; e < 4; ++e) {
            const int64_t jj = j + e;
            if (jj >= end) break;
            while (ly.offsets[li + 1] <= jj) ++li;
            const FmtK& f = spal[ly.fmt_idx ? ly.fmt_idx[li] : 0];
            const int32_t ft = ly.scale_exp ? clamp_exp(ly.scale_exp[li]) : 0;
            const float v = a.Q ? a.Q[jj] : decode(load_code(a.codes, jj, a.code_cls), f);
            a.out[jj] = __builtin_amdgcn_ldexpf(v, -ft);
        }
    }
}

// ================================================== K6: low-precision GEMM

struct GemmArgs {
    const float* __restrict__ A;
    const float* __restrict__ B;
    float* __restrict__ C;
    int64_t lda, ldb, ldc;
    int32_t M, N, K;
    int32_t ka, kb;  // staged A and B carry 2^ka, 2^kb (ka + kb = k of the accumulator, or both 0)
};

// How a product reaches the accumulator's working domain and is rounded:
enum GemmProduct {
    GP_LDEXP = 0,   // operands native: fl32(a * b) then 2^k, rounded (quant)
    GP_SCALED = 1,  // operands pre-scaled at staging: a_w * b_w rounded (quant_w)
    GP_FIT = 2,     // pre-scaled, and every product fits the significand (quant_fit)
};

constexpr int GT = 64;  // output tile GT x GT per block, 4 x 4 per thread
constexpr int GK = 16;  // k-tile staged in LDS

// One block computes a GT x GT tile of C.  Each k-tile of A and B is cast to
// the input format while it is staged into LDS (A transposed, so a thread's
// four rows are one 16-byte read); each thread then runs 16 independent
// chains, one per output, adding its products in k order.  The work is the
// VALU's: a product, its rounding and the rounded add per multiply-accumulate.
template <int V, bool KAHAN, int PM>
__global__ __launch_bounds__(BLOCK) void k_lp_gemm(GemmArgs g, FmtK fi, FmtK fa) {
    __shared__ __align__(16) float As[GK][GT + 4];  // As[k][m]; the pad spreads the staging writes over banks
    __shared__ __align__(16) float Bs[GK][GT + 4];  // Bs[k][n]
    const int t = threadIdx.x;
    const int tx = t & 15, ty = t >> 4;
    const int64_t m0 = (int64_t)blockIdx.y * GT, n0 = (int64_t)blockIdx.x * GT;
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
    // global -> registers, cast to the input format; outside A and B: 0
    auto fetch = [&](int64_t k0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int idx = t + BLOCK * r;
            const int64_t am = m0 + (idx >> 4), ak = k0 + (idx & 15);
            ra[r] = (am < g.M && ak < g.K) ? __builtin_amdgcn_ldexpf(quant_any(g.A[am * g.lda + ak], fi.k, fi), g.ka)
                                           : 0.0f;
            const int64_t bk = k0 + (idx >> 6), bn = n0 + (idx & 63);
            rb[r] = (bk < g.K && bn < g.N) ? __builtin_amdgcn_ldexpf(quant_any(g.B[bk * g.ldb + bn], fi.k, fi), g.kb)
                                           : 0.0f;
        }
    };
    auto mac_v = [&](const f4& av, const f4& bv, bool first) {
        const float a[4] = {av.x, av.y, av.z, av.w};
        const float b[4] = {bv.x, bv.y, bv.z, bv.w};
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
                else
                    p = quant_fit<V>(a[i] * b[j], fa);
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

// ================================================================ host

static int device_cus() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    return cus;
}

static int64_t grid_for(int64_t items, int per_cu) {
    const int cus = device_cus();
    int64_t g = (int64_t)(cus > 0 ? cus : 256) * per_cu;
    if (g > items) g = items;
    return g < 1 ? 1 : g;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

static int check_palette(const aps_format* fmts, int32_t n_fmts, Pal& pal, int* ccls) {
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

static int check_rows(const void* G, int32_t W, int64_t ld, int64_t n, const int64_t* offsets, int32_t L) {
    if (!G || !offsets) return APS_ERR_NULL;
    if (W < 1 || W > APS_MAX_WORKERS || L < 1 || n < 0 || n > APS_MAX_ELEMS || ld < n) return APS_ERR_SIZE;
    if (!aligned16(G) || (ld & 3)) return APS_ERR_ALIGN;
    return APS_OK;
}

static int launched() { return hipGetLastError() == hipSuccess ? APS_OK : APS_ERR_DEVICE; }

// which variants occur in the palette
static unsigned variant_mask(const Pal& pal, int32_t n_fmts) {
    unsigned m = 0;
    for (int i = 0; i < n_fmts; ++i) m |= 1u << pal.f[i].variant;
    return m;
}

}  // namespace aps

using namespace aps;

// The kernels are templates over the variant; dispatch table per entry point.
#define APS_FOR_VARIANTS(X) X(0) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9)

extern "C" int aps_format_supported(aps_format f) { return fmt_status(f); }

extern "C" const char* aps_strerror(int s) {
    switch (s) {
        case APS_OK: return "ok";
        case APS_ERR_NULL: return "required pointer is NULL";
        case APS_ERR_SIZE: return "size argument out of range";
        case APS_ERR_FORMAT: return "format {e, m, bias} out of range";
        case APS_ERR_ALIGN: return "pointer or row stride misaligned";
        case APS_ERR_UNSUPPORTED: return "valid but unsupported combination";
        case APS_ERR_DEVICE: return "HIP launch or device error";
        default: return "unknown status";
    }
}

extern "C" int aps_layer_maxabs(const float* G, int32_t W, int64_t ld, int64_t n, const int64_t* offsets,
                                int32_t L, uint32_t* maxabs_bits, void* stream) {
    int st = check_rows(G, W, ld, n, offsets, L);
    if (st != APS_OK) return st;
    if (!maxabs_bits) return APS_ERR_NULL;
    hipStream_t s = (hipStream_t)stream;
    hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)((L + 255) / 256)), dim3(256), 0, s, maxabs_bits, (int64_t)L, 0u);
    if (n == 0) return launched();
    Layers ly{offsets, nullptr, nullptr, n, L, 1};
    const int64_t nchunks = (n + CH - 1) / CH;
    hipLaunchKernelGGL(k_maxabs, dim3((unsigned)grid_for(nchunks, MAXABS_BLOCKS_PER_CU)), dim3(BLOCK), 0, s, G, W, ld, ly, maxabs_bits);
    return launched();
}

extern "C" int aps_layer_scales(const uint32_t* maxabs_bits, int32_t L, int32_t N, const aps_format* fmts,
                                int32_t n_fmts, const uint8_t* fmt_idx, int32_t* scale_exp, void* stream) {
    if (!maxabs_bits || !scale_exp) return APS_ERR_NULL;
    if (L < 1 || N < 1 || N > APS_MAX_WORKERS) return APS_ERR_SIZE;
    Pal pal;
    int st = check_palette(fmts, n_fmts, pal, nullptr);
    if (st != APS_OK) return st;
    hipLaunchKernelGGL(k_scales, dim3((unsigned)((L + 255) / 256)), dim3(256), 0, (hipStream_t)stream, maxabs_bits,
                       L, N, pal, fmt_idx, scale_exp);
    return launched();
}

extern "C" int aps_quantize(const float* X, int32_t W, int64_t ld, int64_t n, const int64_t* offsets, int32_t L,
                            const int32_t* scale_exp, const aps_format* fmts, int32_t n_fmts,
                            const uint8_t* fmt_idx, float* Q, void* codes, void* stream) {
    int st = check_rows(X, W, ld, n, offsets, L);
    if (st != APS_OK) return st;
    if (!Q && !codes && n > 0) return APS_ERR_NULL;
    if ((Q && !aligned16(Q)) || (codes && !aligned16(codes))) return APS_ERR_ALIGN;
    Pal pal;
    int ccls = 0;
    st = check_palette(fmts, n_fmts, pal, &ccls);
    if (st != APS_OK) return st;
    if (codes && (ccls < 0 || ccls > 2)) return APS_ERR_UNSUPPORTED;
    if (n == 0) return APS_OK;
    hipStream_t s = (hipStream_t)stream;
    Layers ly{offsets, fmt_idx, scale_exp, n, L, n_fmts};
    QuantArgs a{X, Q, (uint8_t*)codes, ld, W, ccls};
    const int64_t nchunks = (n + CH - 1) / CH;
    const dim3 grid((unsigned)grid_for(nchunks, BLOCKS_PER_CU));
    unsigned cm = 0;  // cast variants present
    for (int i = 0; i < n_fmts; ++i) cm |= 1u << cast_variant(pal.f[i].variant);
    const int out = !codes ? QO_Q : (Q ? QO_BOTH : QO_CODES4 + ccls);
#define APS_LAUNCH_Q(v)                                                                                    \
    if (cm & (1u << (v))) {                                                                                \
        switch (out) {                                                                                     \
            case QO_Q: hipLaunchKernelGGL((k_quantize<v, QO_Q>), grid, dim3(BLOCK), 0, s, a, ly, pal); break; \
            case QO_CODES4: hipLaunchKernelGGL((k_quantize<v, QO_CODES4>), grid, dim3(BLOCK), 0, s, a, ly, pal); break; \
            case QO_CODES8: hipLaunchKernelGGL((k_quantize<v, QO_CODES8>), grid, dim3(BLOCK), 0, s, a, ly, pal); break; \
            case QO_CODES16: hipLaunchKernelGGL((k_quantize<v, QO_CODES16>), grid, dim3(BLOCK), 0, s, a, ly, pal); break; \
            default: hipLaunchKernelGGL((k_quantize<v, QO_BOTH>), grid, dim3(BLOCK), 0, s, a, ly, pal); break; \
        }                                                                                                  \
    }
    APS_LAUNCH_Q(V_INT_F64) APS_LAUNCH_Q(V_INT_EXACT) APS_LAUNCH_Q(V_INT_M0) APS_LAUNCH_Q(V_TOP_F64)
    APS_LAUNCH_Q(V_TOP_M0) APS_LAUNCH_Q(V_LOW_F64) APS_LAUNCH_Q(V_LOW_M0)
#undef APS_LAUNCH_Q
    if (fmt_idx && n_fmts > 1 && L > 1)
        hipLaunchKernelGGL(k_quantize_mixed, dim3((unsigned)L, (unsigned)W), dim3(BLOCK), 0, s, a, ly, pal);
    return launched();
}

extern "C" int aps_sim_reduce(const float* G, int32_t W, int64_t ld, int64_t n, const int64_t* offsets,
                              int32_t L, const int32_t* scale_exp, const aps_format* fmts, int32_t n_fmts,
                              const uint8_t* fmt_idx, uint32_t flags, float* out, void* codes_out,
                              void* stream) {
    int st = check_rows(G, W, ld, n, offsets, L);
    if (st != APS_OK) return st;
    if (!out && !codes_out && n > 0) return APS_ERR_NULL;
    if ((out && !aligned16(out)) || (codes_out && !aligned16(codes_out))) return APS_ERR_ALIGN;
    if (flags & ~(APS_INPUT_QUANTIZED | APS_OUTPUT_SCALED)) return APS_ERR_UNSUPPORTED;
    Pal pal;
    int ccls = 0;
    st = check_palette(fmts, n_fmts, pal, &ccls);
    if (st != APS_OK) return st;
    if (codes_out && (ccls < 0 || ccls > 2)) return APS_ERR_UNSUPPORTED;
    if (n == 0) return APS_OK;
    hipStream_t s = (hipStream_t)stream;
    Layers ly{offsets, fmt_idx, scale_exp, n, L, n_fmts};
    ReduceArgs a{G, out, (uint8_t*)codes_out, ld, W, flags, ccls};
    const int64_t nchunks = (n + CH - 1) / CH;
    const dim3 grid((unsigned)grid_for(nchunks, BLOCKS_PER_CU));
    const unsigned vm = variant_mask(pal, n_fmts);
#define APS_LAUNCH_R(v) \
    if (vm & (1u << (v))) hipLaunchKernelGGL(k_sim_reduce<v>, grid, dim3(BLOCK), 0, s, a, ly, pal);
    APS_FOR_VARIANTS(APS_LAUNCH_R)
#undef APS_LAUNCH_R
    if (fmt_idx && n_fmts > 1 && L > 1)
        hipLaunchKernelGGL(k_sim_reduce_mixed, dim3((unsigned)L), dim3(BLOCK), 0, s, a, ly, pal);
    return launched();
}

// Workspace of aps_sync, in 256-byte aligned parts: the per-element exponent
// bytes (padded to whole chunks), four bytes per chunk, the int32 layer
// thresholds, the list counter, the int32 chunk list.
struct SyncLayout {
    uint64_t minb, wmin, thr, count, list, total;
};

static uint64_t up256(uint64_t b) { return (b + 255u) & ~(uint64_t)255u; }

static SyncLayout sync_layout(int64_t n, int32_t L) {
    const uint64_t nch = (uint64_t)((n + CH - 1) / CH);
    SyncLayout o;
    o.minb = 0;
    o.wmin = o.minb + up256(nch * (uint64_t)CH);
    o.thr = o.wmin + up256(4u * nch);
    o.count = o.thr + up256(4u * (uint64_t)L);
    o.list = o.count + 256u;
    o.total = o.list + up256(4u * nch);
    return o;
}

extern "C" uint64_t aps_sync_workspace_bytes(int64_t n, int32_t L) {
    if (n < 0 || L < 0 || n > APS_MAX_ELEMS) return 0;
    return sync_layout(n, L).total;
}

// Which route aps_sync takes.  The one-pass route applies when N = W is a
// power of two (exact N * ghat, no overflow) and every format has m <= 10
// (an fp32 add then one rounding equals rounding the exact sum).  Without a
// route flag it is taken when it is also expected to pay: for layers of
// normally distributed values (max about 5 sigma) an element is recomputed
// with probability about W^2 * 2^(emin - emax + 2), since the threshold sits
// at W * 2^(emin - emax) of the layer's max; above 2^-7 most chunks would be
// recomputed whole and two passes cost less.
static bool sync_one_pass(int32_t W, const Pal& pal, int32_t n_fmts, uint32_t flags) {
    if (flags & APS_SYNC_TWO_PASS) return false;
    if (W & (W - 1)) return false;
    int lw = 0;
    while ((1 << lw) < W) ++lw;
    for (int i = 0; i < n_fmts; ++i) {
        if (pal.f[i].m > 10) return false;
        if (!(flags & APS_SYNC_ONE_PASS) && 2 * lw + pal.f[i].emin - pal.f[i].emax + 2 > -7) return false;
    }
    return true;
}

extern "C" int aps_sync_one_pass(int32_t W, const aps_format* fmts, int32_t n_fmts, uint32_t flags) {
    if (W < 1 || W > APS_MAX_WORKERS) return APS_ERR_SIZE;
    if ((flags & APS_SYNC_ONE_PASS) && (flags & APS_SYNC_TWO_PASS)) return APS_ERR_UNSUPPORTED;
    Pal pal;
    const int st = check_palette(fmts, n_fmts, pal, nullptr);
    if (st != APS_OK) return st;
    return sync_one_pass(W, pal, n_fmts, flags) ? 1 : 0;
}

extern "C" int aps_sync(const float* G, int32_t W, int64_t ld, int64_t n, const int64_t* offsets, int32_t L,
                        const aps_format* fmts, int32_t n_fmts, const uint8_t* fmt_idx, uint32_t flags,
                        uint32_t* maxabs_bits, int32_t* scale_exp, float* out, void* workspace,
                        uint64_t workspace_bytes, void* stream) {
    int st = check_rows(G, W, ld, n, offsets, L);
    if (st != APS_OK) return st;
    if (!maxabs_bits || !scale_exp || !workspace || (!out && n > 0)) return APS_ERR_NULL;
    const uint32_t phases = flags & (APS_SYNC_PASS1 | APS_SYNC_PASS2);
    if (phases == 0 || (flags & ~(APS_SYNC_PASS1 | APS_SYNC_PASS2 | APS_SYNC_ONE_PASS | APS_SYNC_TWO_PASS)) ||
        ((flags & APS_SYNC_ONE_PASS) && (flags & APS_SYNC_TWO_PASS)))
        return APS_ERR_UNSUPPORTED;
    if ((out && !aligned16(out)) || ((uintptr_t)workspace & 255u)) return APS_ERR_ALIGN;
    const SyncLayout lay = sync_layout(n, L);
    if (workspace_bytes < lay.total) return APS_ERR_SIZE;
    Pal pal;
    st = check_palette(fmts, n_fmts, pal, nullptr);
    if (st != APS_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    const int64_t nchunks = (n + CH - 1) / CH;
    uint8_t* wb = (uint8_t*)workspace;
    SyncWs ws{wb + lay.minb, wb + lay.wmin, (int32_t*)(wb + lay.thr), (uint32_t*)(wb + lay.count),
              (int32_t*)(wb + lay.list)};
    Layers ly{offsets, fmt_idx, scale_exp, n, L, n_fmts};
    const bool one = sync_one_pass(W, pal, n_fmts, flags);
    const dim3 lgrid((unsigned)((L + 255) / 256));
    const bool mixed = fmt_idx && n_fmts > 1 && L > 1;
    if (phases & APS_SYNC_PASS1) {
        hipLaunchKernelGGL(k_fill_u32, lgrid, dim3(256), 0, s, maxabs_bits, (int64_t)L, 0u);
        if (n > 0) {
            if (one) {
                SyncArgs sa{G, out, ld, W};
                hipLaunchKernelGGL(k_sync_spec, dim3((unsigned)grid_for(nchunks, BLOCKS_PER_CU)), dim3(BLOCK), 0, s,
                                   sa, ws, ly, pal, maxabs_bits);
            } else {
                Layers lm{offsets, nullptr, nullptr, n, L, 1};
                hipLaunchKernelGGL(k_maxabs, dim3((unsigned)grid_for(nchunks, MAXABS_BLOCKS_PER_CU)), dim3(BLOCK), 0,
                                   s, G, W, ld, lm, maxabs_bits);
            }
        }
    }
    if (phases & APS_SYNC_PASS2) {
        if (!one) {
            hipLaunchKernelGGL(k_scales, lgrid, dim3(256), 0, s, maxabs_bits, L, W, pal, fmt_idx, scale_exp);
            if (n > 0) {
                ReduceArgs a{G, out, nullptr, ld, W, 0u, 0};
                const unsigned vm = variant_mask(pal, n_fmts);
                const dim3 grid((unsigned)grid_for(nchunks, BLOCKS_PER_CU));
#define APS_LAUNCH_R(v) \
    if (vm & (1u << (v))) hipLaunchKernelGGL(k_sim_reduce<v>, grid, dim3(BLOCK), 0, s, a, ly, pal);
                APS_FOR_VARIANTS(APS_LAUNCH_R)
#undef APS_LAUNCH_R
                if (mixed) hipLaunchKernelGGL(k_sim_reduce_mixed, dim3((unsigned)L), dim3(BLOCK), 0, s, a, ly, pal);
            }
        } else {
            hipLaunchKernelGGL(k_sync_layers, lgrid, dim3(256), 0, s, maxabs_bits, L, W, pal, fmt_idx, scale_exp, ws);
            if (n > 0) {
                hipLaunchKernelGGL(k_sync_scan, dim3((unsigned)((nchunks + 255) / 256)), dim3(256), 0, s, ly, ws);
                ReduceArgs a{G, out, nullptr, ld, W, 0u, 0};
                const unsigned vm = variant_mask(pal, n_fmts);
                const dim3 grid((unsigned)grid_for(nchunks, BLOCKS_PER_CU));
#define APS_LAUNCH_S(v) \
    if (vm & (1u << (v))) hipLaunchKernelGGL(k_sync_repair<v>, grid, dim3(BLOCK), 0, s, a, ly, pal, ws);
                APS_LAUNCH_S(V_INT_F32) APS_LAUNCH_S(V_INT_M0) APS_LAUNCH_S(V_TOP_F32) APS_LAUNCH_S(V_TOP_M0)
                APS_LAUNCH_S(V_LOW_F32) APS_LAUNCH_S(V_LOW_M0)
#undef APS_LAUNCH_S
                if (mixed) hipLaunchKernelGGL(k_sync_repair_mixed, dim3((unsigned)L), dim3(BLOCK), 0, s, a, ly, pal, ws);
            }
        }
    }
    return launched();
}

extern "C" int aps_sim_reduce_ex(const float* G, int32_t W, int64_t ld, int64_t n, const int64_t* offsets,
                                 int32_t L, const int32_t* scale_exp, const aps_format* fmts, int32_t n_fmts,
                                 const uint8_t* fmt_idx, uint32_t flags, const aps_reduce_opts* opts, float* out,
                                 void* codes_out, void* stream) {
    const int32_t group = opts ? opts->group : W;
    const int32_t acc = opts ? opts->accumulator : APS_ACC_SEQUENTIAL;
    if (acc != APS_ACC_SEQUENTIAL && acc != APS_ACC_KAHAN) return APS_ERR_UNSUPPORTED;
    if (group < 1 || (group & (group - 1)) != 0 || W % group != 0) {
        // validate the rest first so that the size error is not masked
        const int st = check_rows(G, W, ld, n, offsets, L);
        return st != APS_OK ? st : APS_ERR_SIZE;
    }
    if (group == W && acc == APS_ACC_SEQUENTIAL)
        return aps_sim_reduce(G, W, ld, n, offsets, L, scale_exp, fmts, n_fmts, fmt_idx, flags, out, codes_out,
                              stream);
    int st = check_rows(G, W, ld, n, offsets, L);
    if (st != APS_OK) return st;
    if (!out && !codes_out && n > 0) return APS_ERR_NULL;
    if ((out && !aligned16(out)) || (codes_out && !aligned16(codes_out))) return APS_ERR_ALIGN;
    if (flags & ~(APS_INPUT_QUANTIZED | APS_OUTPUT_SCALED)) return APS_ERR_UNSUPPORTED;
    Pal pal;
    int ccls = 0;
    st = check_palette(fmts, n_fmts, pal, &ccls);
    if (st != APS_OK) return st;
    if (codes_out && (ccls < 0 || ccls > 2)) return APS_ERR_UNSUPPORTED;
    if (n == 0) return APS_OK;
    hipStream_t s = (hipStream_t)stream;
    Layers ly{offsets, fmt_idx, scale_exp, n, L, n_fmts};
    ReduceArgs a{G, out, (uint8_t*)codes_out, ld, W, flags, ccls};
    Order od{__builtin_ctz((unsigned)group), W / group};
    const int64_t nchunks = (n + CH - 1) / CH;
    const dim3 grid((unsigned)grid_for(nchunks, BLOCKS_PER_CU));
    const unsigned vm = variant_mask(pal, n_fmts);
#define APS_LAUNCH_X(v)                                                                                   \
    if (vm & (1u << (v))) {                                                                               \
        if (acc == APS_ACC_KAHAN)                                                                         \
            hipLaunchKernelGGL((k_sim_reduce_ex<v, true>), grid, dim3(BLOCK), 0, s, a, ly, pal, od);     \
        else                                                                                              \
            hipLaunchKernelGGL((k_sim_reduce_ex<v, false>), grid, dim3(BLOCK), 0, s, a, ly, pal, od);    \
    }
    APS_FOR_VARIANTS(APS_LAUNCH_X)
#undef APS_LAUNCH_X
    if (acc == APS_ACC_KAHAN)
        hipLaunchKernelGGL(k_sim_reduce_ex_slow<true>, dim3((unsigned)nchunks), dim3(BLOCK), 0, s, a, ly, pal, od);
    else
        hipLaunchKernelGGL(k_sim_reduce_ex_slow<false>, dim3((unsigned)nchunks), dim3(BLOCK), 0, s, a, ly, pal, od);
    return launched();
}

extern "C" int aps_sim_reduce_codes(const void* codes, int32_t W, int64_t ld, int64_t n, const int64_t* offsets,
                                    int32_t L, const int32_t* scale_exp, const aps_format* fmts, int32_t n_fmts,
                                    const uint8_t* fmt_idx, uint32_t flags, float* out, void* codes_out,
                                    void* stream) {
    if (!codes || !offsets) return APS_ERR_NULL;
    if (W < 1 || W > APS_MAX_WORKERS || L < 1 || n < 0 || n > APS_MAX_ELEMS || ld < n) return APS_ERR_SIZE;
    if (!out && !codes_out && n > 0) return APS_ERR_NULL;
    if (flags & ~APS_OUTPUT_SCALED) return APS_ERR_UNSUPPORTED;
    Pal pal;
    int ccls = 0;
    int st = check_palette(fmts, n_fmts, pal, &ccls);
    if (st != APS_OK) return st;
    if (ccls < 0 || ccls > 2) return APS_ERR_UNSUPPORTED;
    const int64_t row_bytes = code_byte(ld, ccls);
    if (!aligned16(codes) || (row_bytes & 15) || (out && !aligned16(out)) || (codes_out && !aligned16(codes_out)))
        return APS_ERR_ALIGN;
    if (n == 0) return APS_OK;
    hipStream_t s = (hipStream_t)stream;
    Layers ly{offsets, fmt_idx, scale_exp, n, L, n_fmts};
    CodesArgs a{(const uint8_t*)codes, out, (uint8_t*)codes_out, row_bytes, W, flags};
    const int64_t ept = ccls == 0 ? 32 : (ccls == 1 ? 16 : 8);
    const int64_t nchunks = (n + BLOCK * ept - 1) / (BLOCK * ept);
    const dim3 grid((unsigned)grid_for(nchunks, BLOCKS_PER_CU));
    const unsigned vm = variant_mask(pal, n_fmts);
#define APS_LAUNCH_C(v)                                                                                      \
    if (vm & (1u << (v))) {                                                                                  \
        if (ccls == 0) hipLaunchKernelGGL((k_sim_reduce_codes<v, 0>), grid, dim3(BLOCK), 0, s, a, ly, pal);  \
        if (ccls == 1) hipLaunchKernelGGL((k_sim_reduce_codes<v, 1>), grid, dim3(BLOCK), 0, s, a, ly, pal);  \
        if (ccls == 2) hipLaunchKernelGGL((k_sim_reduce_codes<v, 2>), grid, dim3(BLOCK), 0, s, a, ly, pal);  \
    }
    APS_FOR_VARIANTS(APS_LAUNCH_C)
#undef APS_LAUNCH_C
    if (fmt_idx && n_fmts > 1 && L > 1) {
        if (ccls == 0) hipLaunchKernelGGL(k_sim_reduce_codes_mixed<0>, dim3((unsigned)L), dim3(BLOCK), 0, s, a, ly, pal);
        if (ccls == 1) hipLaunchKernelGGL(k_sim_reduce_codes_mixed<1>, dim3((unsigned)L), dim3(BLOCK), 0, s, a, ly, pal);
        if (ccls == 2) hipLaunchKernelGGL(k_sim_reduce_codes_mixed<2>, dim3((unsigned)L), dim3(BLOCK), 0, s, a, ly, pal);
    }
    return launched();
}

extern "C" int aps_dequantize(const float* Q, const void* codes, int64_t n, const int64_t* offsets, int32_t L,
                              const int32_t* scale_exp, const aps_format* fmts, int32_t n_fmts,
                              const uint8_t* fmt_idx, float* out, void* stream) {
    if (!offsets || ((!out || (!Q && !codes)) && n > 0)) return APS_ERR_NULL;
    if (L < 1 || n < 0 || n > APS_MAX_ELEMS) return APS_ERR_SIZE;
    if ((Q && !aligned16(Q)) || (codes && !aligned16(codes)) || !aligned16(out)) return APS_ERR_ALIGN;
    Pal pal;
    int ccls = 0;
    int st = check_palette(fmts, n_fmts, pal, &ccls);
    if (st != APS_OK) return st;
    if (!Q && (ccls < 0 || ccls > 2)) return APS_ERR_UNSUPPORTED;
    if (n == 0) return APS_OK;
    Layers ly{offsets, fmt_idx, scale_exp, n, L, n_fmts};
    DeqArgs a{Q, (const uint8_t*)codes, out, ccls};
    const int64_t nchunks = (n + CH - 1) / CH;
    hipLaunchKernelGGL(k_dequantize, dim3((unsigned)grid_for(nchunks, BLOCKS_PER_CU)), dim3(BLOCK), 0, (hipStream_t)stream, a,
                       ly, pal);
    return launched();
}

// Instantiates only the product modes a variant can take: GP_FIT needs the
// TOP or LOW class with m >= 1; INT-class formats (k = 0) are always scaled.
template <int V>
static void launch_lp_gemm_v(bool kahan, int pm, dim3 grid, hipStream_t s, const GemmArgs& g, const FmtK& fi,
                             const FmtK& fa) {
    constexpr bool can_fit = VT<V>::cls != CLS_INT && !VT<V>::m0;
    constexpr bool can_ldexp = VT<V>::cls != CLS_INT;
#define APS_G(K, P) hipLaunchKernelGGL((k_lp_gemm<V, K, P>), grid, dim3(BLOCK), 0, s, g, fi, fa)
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
    APS_FOR_VARIANTS(APS_LG)
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
    // the product of two input values must be exact in fp32, or round to zero anyway
    const int emin_in = 1 - in_fmt.bias, emin_acc = 1 - acc_fmt.bias;
    if (in_fmt.m > 11) return APS_ERR_UNSUPPORTED;
    if (2 * (emin_in - in_fmt.m) < -149 && 2 * (in_fmt.m + 1) > emin_acc - acc_fmt.m + 149) return APS_ERR_UNSUPPORTED;
    if (!has_out) return APS_OK;
    const FmtK fi = make_fmtk(in_fmt), fa = make_fmtk(acc_fmt);
    GemmArgs g{A, B, C, lda, ldb, ldc, M, N, K, 0, 0};
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
    const dim3 grid((unsigned)((N + GT - 1) / GT), (unsigned)((M + GT - 1) / GT));
    launch_lp_gemm(fa.variant, accumulator == APS_ACC_KAHAN, pm, grid, (hipStream_t)stream, g, fi, fa);
    return launched();
}
