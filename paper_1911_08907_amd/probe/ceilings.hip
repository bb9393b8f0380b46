// ceilings.hip -- what the memory system and the VALU allow the APS kernels,
// measured with the kernels' own access patterns and no arithmetic.
//
// Measurement infrastructure of the benchmark (bench.py --ceilings), built
// into its own library (libaps_probe.so); nothing of the APS path calls it.
// Each probe keeps the launch shape and the load/store pattern of a kernel
// of the path and drops its rounding: a probe's bandwidth is the ceiling that
// pattern sets, and the kernel's own bandwidth divided by it says how much
// the kernel's arithmetic and bookkeeping cost.
//
//   probe_rows   the row walk of k_maxabs / k_sim_reduce / k_sync_spec /
//                k_quantize: per 1024-element chunk, each thread streams its
//                16-byte column slice of all W rows (two register sets of
//                rows in flight), then
//                  READ       keeps an OR of the bits (nothing written),
//                  SUM_F32    writes one fp32 row (the reduced gradient),
//                  SUM_HALF   writes one row of 2-byte halves,
//                  SUM_BYTES  writes one fp32 row and one row of bytes,
//                  ROW_BYTES  writes one byte per element of every row
//                             (aps_quantize to 8-bit codes),
//                  ROW_F32    writes every row back as fp32 (aps_quantize
//                             to values);
//   probe_flat   the same bytes as ROW_BYTES / ROW_F32 in a flat order:
//                each thread reads 16 consecutive elements of one row and
//                writes their 16 bytes (or 64 bytes) at once;
//   probe_rowmajor  the same bytes again, each block walking its chunk range
//                row after row (each row read and written in long runs);
//   probe_rows_wide  the row walk with each block step covering CHX
//                chunks side by side (each thread CHX 16-byte slices of
//                a row, R rows per register set, two sets in flight), so
//                every row is read in runs of CHX * 4 KB;
//   probe_read_flat  a flat read of one contiguous buffer (each block a
//                contiguous range of 16 KB tiles, four 16-byte loads per
//                thread in flight): what HBM gives a pure read stream;
//   probe_copy   a 1:1 fp32 copy, grid-stride (one 16-byte load per thread
//                per step);
//   probe_copy_ranges  the same copy with each block a contiguous range of
//                16 KB tiles, four 16-byte loads per thread in flight;
//   probe_widen  read n codes of `in_bytes` bytes, write n fp32 values
//                (aps_dequantize's traffic), `per` elements per thread;
//   probe_valu   16 independent chains per thread of one VALU instruction.
#include "aps_common.hpp"

namespace aps {
namespace probe {

enum RowMode { READ = 0, SUM_F32 = 1, SUM_HALF = 2, SUM_BYTES = 3, ROW_BYTES = 4, ROW_F32 = 5 };

struct RowArgs {
    const float* __restrict__ G;
    float* __restrict__ out;       // SUM_*: [n]; ROW_F32: [W][ld]
    uint8_t* __restrict__ bytes;   // SUM_BYTES: [n]; ROW_BYTES: [W][ld]
    uint16_t* __restrict__ half;   // SUM_HALF: [n]
    int64_t ld, n;
    int32_t W;
    uint32_t magic;                // never equal to an OR of the data, so READ keeps its loads
};

template <int MODE>
__global__ __launch_bounds__(BLOCK) void k_rows(RowArgs a) {
    const int64_t nchunks = a.n / CH;  // whole chunks only
    int64_t cb, ce;
    block_range(nchunks, cb, ce);
    uint32_t acc = 0;
    for (int64_t c = cb; c < ce; ++c) {
        const int64_t j = c * CH + (int64_t)threadIdx.x * VEC;
        const float* p = a.G + j;
        const int64_t ld = a.ld;
        u4v o = {0u, 0u, 0u, 0u};
        int64_t r = 0;
        auto row = [&](const f4& x, bool valid) {
            if (valid) {
                const u4v b = {f2u(x.x), f2u(x.y), f2u(x.z), f2u(x.w)};
                if constexpr (MODE == ROW_BYTES) {
                    const uint32_t w4 = (b.x >> 24) | ((b.y >> 24) << 8) | ((b.z >> 24) << 16) | (b.w & 0xFF000000u);
                    __builtin_nontemporal_store(w4, (uint32_t*)(a.bytes + r * ld + j));
                } else if constexpr (MODE == ROW_F32) {
                    __builtin_nontemporal_store(x, (f4*)(a.out + r * ld + j));
                } else {
                    o |= b;
                }
            }
            ++r;
        };
        stream_rows(
            a.W, [&](int rr) { return ld4(p + (int64_t)rr * ld); }, [&]() {}, [&](const f4& x) { row(x, true); }, row);
        if constexpr (MODE == READ) acc |= o.x | o.y | o.z | o.w;
        if constexpr (MODE == SUM_F32 || MODE == SUM_BYTES) {
            const f4 v = {u2f(o.x), u2f(o.y), u2f(o.z), u2f(o.w)};
            __builtin_nontemporal_store(v, (f4*)(a.out + j));
        }
        if constexpr (MODE == SUM_BYTES) {
            const uint32_t w4 = (o.x & 0xFFu) | ((o.y & 0xFFu) << 8) | ((o.z & 0xFFu) << 16) | (o.w << 24);
            __builtin_nontemporal_store(w4, (uint32_t*)(a.bytes + j));
        }
        if constexpr (MODE == SUM_HALF) {
            const u2v h = {(o.x >> 16) | (o.y & 0xFFFF0000u), (o.z >> 16) | (o.w & 0xFFFF0000u)};
            __builtin_nontemporal_store(h, (u2v*)(a.half + j));
        }
    }
    if constexpr (MODE == READ)
        if (acc == a.magic) a.out[threadIdx.x] = 1.0f;
}

// Flat order: block b takes a contiguous range of tiles of 4096 elements of
// one row (rows one after another); a thread reads 16 consecutive elements
// and writes their 16 bytes (OUTB = 1) or 64 bytes (OUTB = 4).
template <int OUTB>
__global__ __launch_bounds__(BLOCK) void k_flat(const float* __restrict__ G, uint8_t* __restrict__ dst, int64_t ld,
                                               int64_t n, int32_t W) {
    constexpr int64_t TILE = 16 * BLOCK;
    const int64_t tpr = n / TILE;  // whole tiles per row
    int64_t tb, te;
    block_range(tpr * W, tb, te);
    for (int64_t t = tb; t < te; ++t) {
        const int64_t w = t / tpr;
        const int64_t j = (t - w * tpr) * TILE + 16 * (int64_t)threadIdx.x;
        const float* p = G + w * ld + j;
        f4 x[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) x[k] = ld4(p + 4 * k);
        if constexpr (OUTB == 1) {
            u4v c;
#pragma unroll
            for (int k = 0; k < 4; ++k)
                c[k] = (f2u(x[k].x) >> 24) | ((f2u(x[k].y) >> 24) << 8) | ((f2u(x[k].z) >> 24) << 16) |
                       (f2u(x[k].w) & 0xFF000000u);
            __builtin_nontemporal_store(c, (u4v*)(dst + w * ld + j));
        } else {
#pragma unroll
            for (int k = 0; k < 4; ++k) __builtin_nontemporal_store(x[k], (f4*)((float*)dst + w * ld + j + 4 * k));
        }
    }
}

// Row-major order inside a block's range of chunks: for each row, the block
// walks all its chunks (G of them in flight), so each row is read and
// written in one long run; OUTB = 1 writes a byte per element, 4 an fp32.
template <int OUTB, int G>
__global__ __launch_bounds__(BLOCK) void k_rowmajor(const float* __restrict__ X, uint8_t* __restrict__ dst, int64_t ld,
                                                   int64_t n, int32_t W) {
    const int64_t nchunks = n / CH;  // whole chunks only
    int64_t cb, ce;
    block_range(nchunks, cb, ce);
    for (int64_t w = 0; w < W; ++w) {
        for (int64_t c0 = cb; c0 < ce; c0 += G) {
            f4 x[G];
#pragma unroll
            for (int g = 0; g < G; ++g)
                if (c0 + g < ce) x[g] = ld4(X + w * ld + (c0 + g) * CH + (int64_t)threadIdx.x * VEC);
#pragma unroll
            for (int g = 0; g < G; ++g) {
                if (c0 + g >= ce) break;
                const int64_t j = (c0 + g) * CH + (int64_t)threadIdx.x * VEC;
                if constexpr (OUTB == 1) {
                    const uint32_t w4 = (f2u(x[g].x) >> 24) | ((f2u(x[g].y) >> 24) << 8) | ((f2u(x[g].z) >> 24) << 16) |
                                        (f2u(x[g].w) & 0xFF000000u);
                    __builtin_nontemporal_store(w4, (uint32_t*)(dst + w * ld + j));
                } else {
                    __builtin_nontemporal_store(x[g], (f4*)((float*)dst + w * ld + j));
                }
            }
        }
    }
}

// Flat order with coalesced loads: block b takes a contiguous range of tiles
// of 4 chunks of one row (rows one after another); per tile each thread
// loads its 16-byte slice of the 4 chunks and writes the 4 code bytes of
// each (4 stores of 4 bytes, STAGED = 0), or passes them through LDS so
// that it stores 16 consecutive code bytes at once (STAGED = 1).
template <int STAGED>
__global__ __launch_bounds__(BLOCK) void k_flatrow_bytes(const float* __restrict__ G, uint8_t* __restrict__ dst,
                                                        int64_t ld, int64_t row_bytes, int64_t n, int32_t W) {
    __shared__ uint32_t lds[4 * BLOCK];
    constexpr int64_t TILE = 4 * CH;
    const int64_t tpr = n / TILE;  // whole tiles per row
    int64_t tb, te;
    block_range(tpr * W, tb, te);
    for (int64_t t = tb; t < te; ++t) {
        const int64_t w = t / tpr;
        const int64_t j0 = (t - w * tpr) * TILE;
        const float* p = G + w * ld + j0 + (int64_t)threadIdx.x * VEC;
        f4 x[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) x[k] = ld4(p + k * CH);
        uint32_t c[4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
            c[k] = (f2u(x[k].x) >> 24) | ((f2u(x[k].y) >> 24) << 8) | ((f2u(x[k].z) >> 24) << 16) |
                   (f2u(x[k].w) & 0xFF000000u);
        uint8_t* d = dst + w * row_bytes + j0;
        if constexpr (STAGED == 0) {
#pragma unroll
            for (int k = 0; k < 4; ++k)
                __builtin_nontemporal_store(c[k], (uint32_t*)(d + k * CH + (int64_t)threadIdx.x * VEC));
        } else {
#pragma unroll
            for (int k = 0; k < 4; ++k) lds[k * BLOCK + threadIdx.x] = c[k];
            __syncthreads();
            const u4v v = {lds[4 * threadIdx.x], lds[4 * threadIdx.x + 1], lds[4 * threadIdx.x + 2],
                           lds[4 * threadIdx.x + 3]};
            __syncthreads();
            __builtin_nontemporal_store(v, (u4v*)(d + 16 * (int64_t)threadIdx.x));
        }
    }
}

__global__ __launch_bounds__(BLOCK) void k_copy(const f4* __restrict__ src, f4* __restrict__ dst, int64_t n4) {
    const int64_t stride = (int64_t)gridDim.x * BLOCK;
    for (int64_t i = (int64_t)blockIdx.x * BLOCK + threadIdx.x; i < n4; i += stride)
        __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

// The row walk with CHX chunks per block step: thread t owns the 16-byte
// slice at element 4t of each of the CHX chunks; R rows per register set,
// two sets in flight (W a multiple of 2R).  OUT_NONE keeps an OR of the
// bits, OUT_HALF writes one row of 2-byte halves, OUT_F32 one fp32 row.
enum WideOut { OUT_NONE = 0, OUT_HALF = 1, OUT_F32 = 2 };

template <int CHX, int R, int OUT>
__global__ __launch_bounds__(BLOCK) void k_rows_wide(RowArgs a) {
    constexpr int64_t C = CHX * CH;
    int64_t gb, ge;
    block_range(a.n / C, gb, ge);
    u4v keep = {0u, 0u, 0u, 0u};
    const int K = a.W / (2 * R);  // pairs of register sets
    for (int64_t g = gb; g < ge; ++g) {
        const int64_t j = g * C + (int64_t)threadIdx.x * VEC;
        const float* p = a.G + j;
        const int64_t ld = a.ld;
        u4v acc[CHX];
        f4 A[R][CHX], B[R][CHX];
#pragma unroll
        for (int u = 0; u < CHX; ++u) acc[u] = (u4v){0u, 0u, 0u, 0u};
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int u = 0; u < CHX; ++u) A[r][u] = ld4(p + (int64_t)r * ld + u * CH);
        for (int k = 0; k + 1 < K; ++k) {
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int u = 0; u < CHX; ++u) B[r][u] = ld4(p + (int64_t)(2 * k * R + R + r) * ld + u * CH);
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int u = 0; u < CHX; ++u) acc[u] |= __builtin_bit_cast(u4v, A[r][u]);
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int u = 0; u < CHX; ++u) A[r][u] = ld4(p + (int64_t)(2 * k * R + 2 * R + r) * ld + u * CH);
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int u = 0; u < CHX; ++u) acc[u] |= __builtin_bit_cast(u4v, B[r][u]);
        }
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int u = 0; u < CHX; ++u) B[r][u] = ld4(p + (int64_t)(a.W - R + r) * ld + u * CH);
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int u = 0; u < CHX; ++u) acc[u] |= __builtin_bit_cast(u4v, A[r][u]) | __builtin_bit_cast(u4v, B[r][u]);
#pragma unroll
        for (int u = 0; u < CHX; ++u) {
            const int64_t jj = j + u * CH;
            const u4v o = acc[u];
            if constexpr (OUT == OUT_NONE) keep |= o;
            if constexpr (OUT == OUT_F32)
                __builtin_nontemporal_store(__builtin_bit_cast(f4, o), (f4*)(a.out + jj));
            if constexpr (OUT == OUT_HALF) {
                const u2v h = {(o.x >> 16) | (o.y & 0xFFFF0000u), (o.z >> 16) | (o.w & 0xFFFF0000u)};
                __builtin_nontemporal_store(h, (u2v*)(a.half + jj));
            }
        }
    }
    if constexpr (OUT == OUT_NONE)
        if ((keep.x | keep.y | keep.z | keep.w) == a.magic) a.out[threadIdx.x] = 1.0f;
}

// A flat read of n4 16-byte items: each block a contiguous range of tiles of
// 4 * BLOCK items, four loads per thread in flight.
__global__ __launch_bounds__(BLOCK) void k_read_flat(const f4* __restrict__ src, int64_t n4, float* __restrict__ sink,
                                                    uint32_t magic) {
    int64_t tb, te;
    block_range(n4 / (4 * BLOCK), tb, te);
    u4v acc = {0u, 0u, 0u, 0u};
    for (int64_t t = tb; t < te; ++t) {
        const f4* p = src + t * 4 * BLOCK + threadIdx.x;
        f4 x[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) x[u] = __builtin_nontemporal_load(p + u * BLOCK);
#pragma unroll
        for (int u = 0; u < 4; ++u) acc |= __builtin_bit_cast(u4v, x[u]);
    }
    if ((acc.x | acc.y | acc.z | acc.w) == magic) sink[threadIdx.x] = 1.0f;
}

// The copy in the same order: tiles of 4 * BLOCK items per block step.
__global__ __launch_bounds__(BLOCK) void k_copy_ranges(const f4* __restrict__ src, f4* __restrict__ dst, int64_t n4) {
    int64_t tb, te;
    block_range(n4 / (4 * BLOCK), tb, te);
    for (int64_t t = tb; t < te; ++t) {
        const int64_t i = t * 4 * BLOCK + threadIdx.x;
        f4 x[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) x[u] = __builtin_nontemporal_load(src + i + u * BLOCK);
#pragma unroll
        for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(x[u], dst + i + u * BLOCK);
    }
}

// n codes of IN bytes each in, n fp32 out; PER elements per thread per step.
template <int IN, int PER>
__global__ __launch_bounds__(BLOCK) void k_widen(const uint8_t* __restrict__ in, float* __restrict__ out, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * BLOCK * PER;
    for (int64_t j = ((int64_t)blockIdx.x * BLOCK + threadIdx.x) * PER; j + PER <= n; j += stride) {
        uint32_t w[PER * IN / 4 > 0 ? PER * IN / 4 : 1];
        if constexpr (PER * IN == 4) {
            w[0] = __builtin_nontemporal_load((const uint32_t*)(in + j * IN));
        } else if constexpr (PER * IN == 8) {
            const u2v v = __builtin_nontemporal_load((const u2v*)(in + j * IN));
            w[0] = v.x;
            w[1] = v.y;
        } else {
#pragma unroll
            for (int k = 0; k < PER * IN / 16; ++k) {
                const u4v v = __builtin_nontemporal_load((const u4v*)(in + j * IN) + k);
                w[4 * k] = v.x;
                w[4 * k + 1] = v.y;
                w[4 * k + 2] = v.z;
                w[4 * k + 3] = v.w;
            }
        }
#pragma unroll
        for (int k = 0; k < PER / 4; ++k) {
            f4 o;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int idx = 4 * k + e;  // element within the thread's run
                const uint32_t word = w[idx * IN / 4];
                const uint32_t code = IN == 1 ? (word >> (8 * (idx & 3))) & 0xFFu : (word >> (16 * (idx & 1))) & 0xFFFFu;
                o[e] = u2f(code << (IN == 1 ? 24 : 16));
            }
            __builtin_nontemporal_store(o, (f4*)(out + j) + k);
        }
    }
}

enum ValuOp { V_ADD = 0, V_MUL = 1, V_AND = 2, V_FMA = 3, V_ADD3 = 4, V_BFE = 5, V_LDEXP = 6, V_AND_OR = 7,
              V_SUBREV = 8, V_CMP_CNDMASK = 9, V_CMP_CNDMASK_SGPR = 10, V_RNDNE = 11,
              V_PK_ADD_F16 = 12, V_PK_MUL_F16 = 13, V_CVT_PK_BF16 = 14 };

template <int OP>
__device__ __forceinline__ void valu_step(float& x, float y, float z, int s) {
    if constexpr (OP == V_ADD) asm volatile("v_add_f32_e32 %0, %1, %0" : "+v"(x) : "v"(y));
    if constexpr (OP == V_MUL) asm volatile("v_mul_f32_e32 %0, %1, %0" : "+v"(x) : "v"(y));
    if constexpr (OP == V_AND) asm volatile("v_and_b32_e32 %0, %1, %0" : "+v"(x) : "v"(y));
    if constexpr (OP == V_FMA) asm volatile("v_fma_f32 %0, %1, %2, %0" : "+v"(x) : "v"(y), "v"(z));
    if constexpr (OP == V_ADD3) asm volatile("v_add3_u32 %0, %1, %2, %0" : "+v"(x) : "v"(y), "v"(z));
    if constexpr (OP == V_BFE) asm volatile("v_bfe_u32 %0, %0, %1, %2" : "+v"(x) : "v"(y), "v"(z));
    if constexpr (OP == V_LDEXP) asm volatile("v_ldexp_f32 %0, %0, %1" : "+v"(x) : "v"(s));
    if constexpr (OP == V_AND_OR) asm volatile("v_and_or_b32 %0, %0, %1, %2" : "+v"(x) : "v"(y), "v"(z));
    if constexpr (OP == V_SUBREV) asm volatile("v_subrev_f32_e32 %0, %1, %0" : "+v"(x) : "v"(y));
    if constexpr (OP == V_RNDNE) asm volatile("v_rndne_f32_e32 %0, %0" : "+v"(x));
    // packed half precision: two lanes of work per instruction (counted as one instruction)
    if constexpr (OP == V_PK_ADD_F16) asm volatile("v_pk_add_f16 %0, %1, %0" : "+v"(x) : "v"(y));
    if constexpr (OP == V_PK_MUL_F16) asm volatile("v_pk_mul_f16 %0, %1, %0" : "+v"(x) : "v"(y));
    // two fp32 values to a pair of bfloat16 (counted as one instruction)
    if constexpr (OP == V_CVT_PK_BF16) asm volatile("v_cvt_pk_bf16_f32 %0, %0, %1" : "+v"(x) : "v"(y));
    // a compare into VCC and a select by it, as the compiler emits a rounding's
    // branch-free choice (one pair counted as two instructions)
    if constexpr (OP == V_CMP_CNDMASK)
        asm volatile("v_cmp_nle_f32_e32 vcc, %0, %1\n\tv_cndmask_b32_e32 %0, %1, %0, vcc" : "+v"(x) : "v"(y) : "vcc");
    // the same pair with the mask in an SGPR pair of its own (VOP3 forms)
    if constexpr (OP == V_CMP_CNDMASK_SGPR) {
        uint64_t m;
        asm volatile("v_cmp_nle_f32_e64 %1, %0, %2\n\tv_cndmask_b32_e64 %0, %2, %0, %1" : "+v"(x), "=&s"(m) : "v"(y));
    }
}

template <int OP>
__global__ __launch_bounds__(BLOCK) void k_valu(float* __restrict__ out, int32_t iters, uint32_t magic) {
    float v[16];
    const float y = u2f(0x3F800001u ^ threadIdx.x), z = u2f(0x00000003u);
    const int s = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) v[k] = u2f(0x3F800000u + (uint32_t)(k * 977 + threadIdx.x));
#pragma unroll 1
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
#pragma unroll
            for (int k = 0; k < 16; ++k) valu_step<OP>(v[k], y, z, s);
        }
    }
    uint32_t acc = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) acc ^= f2u(v[k]);
    if (acc == magic) out[threadIdx.x] = 1.0f;
}

}  // namespace probe
}  // namespace aps

using namespace aps;
using namespace aps::probe;

static int probe_done() { return hipGetLastError() == hipSuccess ? 0 : -6; }

// mode: RowMode; blocks_per_cu: launch width (the path's kernels use 24 per
// CU from 64 rows on, 32 below); n: elements per row, whole 1024-element
// chunks are walked.
extern "C" int probe_rows(int mode, const float* G, int32_t W, int64_t ld, int64_t n, float* out, void* bytes,
                          void* half, int blocks_per_cu, void* stream) {
    if (!G || W < 1 || n < CH || ld < n || (ld & 3) || blocks_per_cu < 1) return -2;
    RowArgs a{G, out, (uint8_t*)bytes, (uint16_t*)half, ld, n, W, 0x5A5A5A5Au};
    const dim3 grid((unsigned)grid_for(n / CH, blocks_per_cu));
    hipStream_t s = (hipStream_t)stream;
    switch (mode) {
        case READ: hipLaunchKernelGGL(k_rows<READ>, grid, dim3(BLOCK), 0, s, a); break;
        case SUM_F32: hipLaunchKernelGGL(k_rows<SUM_F32>, grid, dim3(BLOCK), 0, s, a); break;
        case SUM_HALF: hipLaunchKernelGGL(k_rows<SUM_HALF>, grid, dim3(BLOCK), 0, s, a); break;
        case SUM_BYTES: hipLaunchKernelGGL(k_rows<SUM_BYTES>, grid, dim3(BLOCK), 0, s, a); break;
        case ROW_BYTES: hipLaunchKernelGGL(k_rows<ROW_BYTES>, grid, dim3(BLOCK), 0, s, a); break;
        case ROW_F32: hipLaunchKernelGGL(k_rows<ROW_F32>, grid, dim3(BLOCK), 0, s, a); break;
        default: return -5;
    }
    return probe_done();
}

// outb: 1 (bytes) or 4 (fp32); dst is [W][ld] of that element size.
extern "C" int probe_flat(int outb, const float* G, int32_t W, int64_t ld, int64_t n, void* dst, int blocks_per_cu,
                          void* stream) {
    if (!G || !dst || W < 1 || n < 16 * BLOCK || ld < n || (ld & 15) || blocks_per_cu < 1) return -2;
    const int64_t tiles = (n / (16 * BLOCK)) * W;
    const dim3 grid((unsigned)grid_for(tiles, blocks_per_cu));
    hipStream_t s = (hipStream_t)stream;
    if (outb == 1)
        hipLaunchKernelGGL(k_flat<1>, grid, dim3(BLOCK), 0, s, G, (uint8_t*)dst, ld, n, W);
    else if (outb == 4)
        hipLaunchKernelGGL(k_flat<4>, grid, dim3(BLOCK), 0, s, G, (uint8_t*)dst, ld, n, W);
    else
        return -5;
    return probe_done();
}

// Row-major walk (k_rowmajor): outb 1 or 4, g chunks in flight (1, 4 or 8).
extern "C" int probe_rowmajor(int outb, int g, const float* X, int32_t W, int64_t ld, int64_t n, void* dst,
                              int blocks_per_cu, void* stream) {
    if (!X || !dst || W < 1 || n < CH || ld < n || (ld & 3) || blocks_per_cu < 1) return -2;
    const dim3 grid((unsigned)grid_for(n / CH, blocks_per_cu));
    hipStream_t s = (hipStream_t)stream;
    uint8_t* d = (uint8_t*)dst;
#define PROBE_RM(O, GG) \
    if (outb == O && g == GG) { hipLaunchKernelGGL((k_rowmajor<O, GG>), grid, dim3(BLOCK), 0, s, X, d, ld, n, W); return probe_done(); }
    PROBE_RM(1, 1) PROBE_RM(1, 4) PROBE_RM(1, 8) PROBE_RM(4, 1) PROBE_RM(4, 4) PROBE_RM(4, 8)
#undef PROBE_RM
    return -5;
}

extern "C" int probe_copy(const float* src, float* dst, int64_t n, int blocks_per_cu, void* stream) {
    if (!src || !dst || n < 4 || (n & 3) || blocks_per_cu < 1) return -2;
    const int64_t n4 = n / 4;
    hipLaunchKernelGGL(k_copy, dim3((unsigned)grid_for((n4 + BLOCK - 1) / BLOCK, blocks_per_cu)), dim3(BLOCK), 0,
                       (hipStream_t)stream, (const f4*)src, (f4*)dst, n4);
    return probe_done();
}

// The wide row walk: chx chunks per block step (2 or 4), r rows per register
// set (2 or 4), out 0 (read only), 1 (2-byte halves) or 2 (fp32 row); W a
// multiple of 2r; whole steps of chx chunks are walked.
extern "C" int probe_rows_wide(int chx, int r, int out_mode, const float* G, int32_t W, int64_t ld, int64_t n,
                               float* out, void* half, int blocks_per_cu, void* stream) {
    if (!G || !out || W < 1 || (W % (2 * r)) || n < chx * CH || ld < n || (ld & 3) || blocks_per_cu < 1) return -2;
    if (out_mode == OUT_HALF && !half) return -2;
    RowArgs a{G, out, nullptr, (uint16_t*)half, ld, n, W, 0x5A5A5A5Au};
    const dim3 grid((unsigned)grid_for(n / (chx * CH), blocks_per_cu));
    hipStream_t s = (hipStream_t)stream;
#define PROBE_RW(X, RR, O)                                                                  \
    if (chx == X && r == RR && out_mode == O) {                                             \
        hipLaunchKernelGGL((k_rows_wide<X, RR, O>), grid, dim3(BLOCK), 0, s, a);            \
        return probe_done();                                                                \
    }
    PROBE_RW(2, 2, OUT_NONE) PROBE_RW(2, 2, OUT_HALF) PROBE_RW(2, 2, OUT_F32)
    PROBE_RW(2, 4, OUT_NONE) PROBE_RW(2, 4, OUT_HALF) PROBE_RW(2, 4, OUT_F32)
    PROBE_RW(4, 2, OUT_NONE) PROBE_RW(4, 2, OUT_HALF) PROBE_RW(4, 2, OUT_F32)
#undef PROBE_RW
    return -5;
}

// A flat read of n floats (n a multiple of 4 * 4 * BLOCK); sink needs BLOCK floats.
extern "C" int probe_read_flat(const float* src, int64_t n, float* sink, int blocks_per_cu, void* stream) {
    if (!src || !sink || n < 16 * BLOCK || (n % (16 * BLOCK)) || blocks_per_cu < 1) return -2;
    const int64_t n4 = n / 4;
    hipLaunchKernelGGL(k_read_flat, dim3((unsigned)grid_for(n4 / (4 * BLOCK), blocks_per_cu)), dim3(BLOCK), 0,
                       (hipStream_t)stream, (const f4*)src, n4, sink, 0x5A5A5A5Au);
    return probe_done();
}

// The copy of n floats in block ranges (n a multiple of 4 * 4 * BLOCK).
extern "C" int probe_copy_ranges(const float* src, float* dst, int64_t n, int blocks_per_cu, void* stream) {
    if (!src || !dst || n < 16 * BLOCK || (n % (16 * BLOCK)) || blocks_per_cu < 1) return -2;
    const int64_t n4 = n / 4;
    hipLaunchKernelGGL(k_copy_ranges, dim3((unsigned)grid_for(n4 / (4 * BLOCK), blocks_per_cu)), dim3(BLOCK), 0,
                       (hipStream_t)stream, (const f4*)src, (f4*)dst, n4);
    return probe_done();
}

// Flat coalesced walk writing a byte per element (k_flatrow_bytes): staged 0
// or 1; n a multiple of 4 chunks, ld >= n, row_bytes >= n.
extern "C" int probe_flatrow_bytes(int staged, const float* G, int32_t W, int64_t ld, int64_t n, void* dst,
                                   int64_t row_bytes, int blocks_per_cu, void* stream) {
    if (!G || !dst || W < 1 || n < 4 * CH || (n % (4 * CH)) || ld < n || row_bytes < n || blocks_per_cu < 1) return -2;
    const dim3 grid((unsigned)grid_for(n / (4 * CH) * W, blocks_per_cu));
    hipStream_t s = (hipStream_t)stream;
    if (staged == 0)
        hipLaunchKernelGGL(k_flatrow_bytes<0>, grid, dim3(BLOCK), 0, s, G, (uint8_t*)dst, ld, row_bytes, n, W);
    else if (staged == 1)
        hipLaunchKernelGGL(k_flatrow_bytes<1>, grid, dim3(BLOCK), 0, s, G, (uint8_t*)dst, ld, row_bytes, n, W);
    else
        return -5;
    return probe_done();
}

// in_bytes: 1 or 2; per: 4 or 16 elements per thread; n a multiple of per.
extern "C" int probe_widen(int in_bytes, int per, const void* in, float* out, int64_t n, int blocks_per_cu,
                           void* stream) {
    if (!in || !out || n < per || blocks_per_cu < 1) return -2;
    const dim3 grid((unsigned)grid_for((n / per + BLOCK - 1) / BLOCK, blocks_per_cu));
    hipStream_t s = (hipStream_t)stream;
    const uint8_t* p = (const uint8_t*)in;
    if (in_bytes == 1 && per == 4) hipLaunchKernelGGL((k_widen<1, 4>), grid, dim3(BLOCK), 0, s, p, out, n);
    else if (in_bytes == 1 && per == 16) hipLaunchKernelGGL((k_widen<1, 16>), grid, dim3(BLOCK), 0, s, p, out, n);
    else if (in_bytes == 2 && per == 4) hipLaunchKernelGGL((k_widen<2, 4>), grid, dim3(BLOCK), 0, s, p, out, n);
    else if (in_bytes == 2 && per == 16) hipLaunchKernelGGL((k_widen<2, 16>), grid, dim3(BLOCK), 0, s, p, out, n);
    else return -5;
    return probe_done();
}

// op: ValuOp; every thread runs iters * 64 instructions of that kind (16
// independent chains); out needs BLOCK floats.
extern "C" int probe_valu(int op, float* out, int blocks_per_cu, int32_t iters, void* stream) {
    if (!out || blocks_per_cu < 1 || iters < 1) return -2;
    const dim3 grid((unsigned)grid_for((int64_t)1 << 30, blocks_per_cu));
    hipStream_t s = (hipStream_t)stream;
    const uint32_t magic = 0x12345678u;
#define PROBE_V(o) \
    case o: hipLaunchKernelGGL(k_valu<o>, grid, dim3(BLOCK), 0, s, out, iters, magic); break;
    switch (op) {
        PROBE_V(V_ADD) PROBE_V(V_MUL) PROBE_V(V_AND) PROBE_V(V_FMA) PROBE_V(V_ADD3) PROBE_V(V_BFE) PROBE_V(V_LDEXP)
        PROBE_V(V_AND_OR) PROBE_V(V_SUBREV) PROBE_V(V_CMP_CNDMASK) PROBE_V(V_CMP_CNDMASK_SGPR) PROBE_V(V_RNDNE)
        PROBE_V(V_PK_ADD_F16) PROBE_V(V_PK_MUL_F16) PROBE_V(V_CVT_PK_BF16)
        default: return -5;
    }
#undef PROBE_V
    return probe_done();
}

// Compute units of the current device (the grids above are per CU).
extern "C" int probe_device_cus(void) { return device_cus(); }
