// aps_core.hip -- the step's kernels and their C ABI entry points: per-layer
// max magnitude (FindMaxExp input + AllReduce MAX), power-of-two scale
// exponents (Sec. 3.3.3), and the fused scale + cast + SUM all-reduce with a
// low-precision accumulator rounded after every add in worker order + cast
// back + unscale (Algorithm 1; Sec. 3.3.1, Sec. 4, Sec. 5).
#include "aps_common.hpp"

namespace aps {

// ============================================================ K0: fill

__global__ void k_fill_u32(uint32_t* __restrict__ p, int64_t cnt, uint32_t v) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < cnt) p[i] = v;
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

// ST: the outputs go through an LDS stage (no codes written).
template <int V, bool ST>
__global__ __launch_bounds__(BLOCK) void k_sim_reduce(ReduceArgs a, Layers ly, Pal pal) {
    __shared__ f4 st_o[ST ? OUT_STAGE * BLOCK : 1];
    __shared__ int32_t st_j[ST ? OUT_STAGE * BLOCK : 1];
    __shared__ int32_t st_lim[ST ? OUT_STAGE * BLOCK : 1];
    OutStage stage{st_o, st_j, st_lim, 0};
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
        if constexpr (ST) drain_if_full(a, stage);
        reduce_vec<V>(a, f, j, end, ft, pd, nullptr, ST ? &stage : nullptr);
    }
    if constexpr (ST) {
        drain_if_full(a, stage);
        stage_out(pd, stage);
        drain_out(a, stage);
    } else {
        flush_out(a, pd);
    }
}

// Chunks whose layers use different palette entries, element by element.
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

}  // namespace aps

using namespace aps;

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
    const dim3 grid((unsigned)stream_grid(nchunks, W, BLOCKS_PER_CU));
    const unsigned vm = variant_mask(pal, n_fmts);
#define APS_LAUNCH_R(v)                                                                             \
    if (vm & (1u << (v))) {                                                                         \
        if (codes_out)                                                                              \
            hipLaunchKernelGGL((k_sim_reduce<v, false>), grid, dim3(BLOCK), 0, s, a, ly, pal);       \
        else                                                                                        \
            hipLaunchKernelGGL((k_sim_reduce<v, true>), grid, dim3(BLOCK), 0, s, a, ly, pal);        \
    }
    APS_FOR_VARIANTS(APS_LAUNCH_R)
#undef APS_LAUNCH_R
    if (fmt_idx && n_fmts > 1 && L > 1)
        hipLaunchKernelGGL(k_sim_reduce_mixed, dim3((unsigned)L), dim3(BLOCK), 0, s, a, ly, pal);
    return launched();
}
