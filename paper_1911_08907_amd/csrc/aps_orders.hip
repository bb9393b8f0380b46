// aps_orders.hip -- the W-worker rounded sum in the order of the
// hierarchical all-reduce of Sec. 4.2 (groups, ring over the masters), with
// the plain or Kahan low-precision accumulator of Sec. 5.
#include "aps_common.hpp"

namespace aps {

// ======================================= K4x: summation orders, Kahan

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
        // chunks that mix palette entries: k_sim_reduce_ex_slow; chunks that
        // cross ring segments: k_sim_reduce_ex_cross
        if (ci.mixed || seg != ring_segment(end - 1, ly.n, od.ng)) continue;
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

// Chunks of one palette entry that cross ring segments, one block per
// segment boundary (the block of the first boundary inside a chunk owns it):
// one row walk per segment the chunk touches; after each, the elements of
// that segment are stored at once (a thread owns both nibbles of its code
// bytes, so the read-modify-writes of a byte split between segments come in
// program order).  A kernel of its own, so that the usual chunk keeps the
// register footprint of a single walk.
template <int V, bool KAHAN>
__global__ __launch_bounds__(BLOCK) void k_sim_reduce_ex_cross(ReduceArgs a, Layers ly, Pal pal, Order od) {
    const int64_t s1 = (int64_t)blockIdx.x + 1;                // boundary: first element of segment s1
    const int64_t p = (s1 * ly.n + od.ng - 1) / od.ng;
    if (p <= 0 || p >= ly.n || p % CH == 0) return;           // at a chunk edge: nothing crosses
    const int64_t start = p / CH * CH;
    if (s1 > 1 && ((s1 - 1) * ly.n + od.ng - 1) / od.ng > start) return;  // an earlier boundary owns it
    const int64_t end = min(start + CH, ly.n);
    const ChunkInfo ci = chunk_layers(ly, start, end, 0);
    if (ci.mixed) return;  // k_sim_reduce_ex_slow
    const FmtK& f = pal.f[ci.pidx];
    if (f.variant != V) return;
    const int64_t j = start + (int64_t)threadIdx.x * VEC;
    if (j >= end) return;
    int32_t ft[4];
    if (ci.i0 == ci.i1) {
        const int32_t t = ly.scale_exp ? clamp_exp(cld(ly.scale_exp, ci.i0)) : 0;
        ft[0] = ft[1] = ft[2] = ft[3] = t;
    } else {
        elem_scales(ly, ci, j, ft);
    }
    const int64_t seg_last = ring_segment(end - 1, ly.n, od.ng);
    for (int64_t sg = ring_segment(start, ly.n, od.ng); sg <= seg_last; ++sg) {
        PendingOut part;
        part.valid = false;
        reduce_vec_ex<V, KAHAN>(a, f, j, end, ft, (int)sg, od, part);
        // segment sg holds the elements i with floor(i * ng / n) = sg
        const int64_t lo = (sg * ly.n + od.ng - 1) / od.ng;
        const int64_t hi = min(((sg + 1) * ly.n + od.ng - 1) / od.ng, end);
        const float po[4] = {part.o.x, part.o.y, part.o.z, part.o.w};
        for (int e = 0; e < 4; ++e) {
            const int64_t jj = j + e;
            if (jj < lo || jj >= hi) continue;
            if (a.out) a.out[jj] = po[e];
            if (a.codes) {
                if (a.code_cls == 0) {
                    uint8_t* pb = a.codes + (jj >> 1);
                    *pb = (jj & 1) ? (uint8_t)((*pb & 0x0Fu) | ((part.c[e] & 15u) << 4))
                                   : (uint8_t)((*pb & 0xF0u) | (part.c[e] & 15u));
                } else {
                    put_code(a.codes, jj, part.c[e], a.code_cls);
                }
            }
        }
    }
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
        case V_GEN: return reduce_elem_ex<V_GEN, KAHAN>(a, f, j, F, seg, od);
        default: return reduce_elem_ex<V_LOW_M0, KAHAN>(a, f, j, F, seg, od);
    }
}

// Chunks that mix palette entries, one block per chunk (blocks of other
// chunks return at once); element pairs per thread so that a byte of nibble
// codes has one writer.
template <bool KAHAN>
__global__ __launch_bounds__(BLOCK) void k_sim_reduce_ex_slow(ReduceArgs a, Layers ly, Pal pal, Order od) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    const int64_t start = (int64_t)blockIdx.x * CH;
    if (start >= ly.n) return;
    const int64_t end = min(start + CH, ly.n);
    const ChunkInfo ci = chunk_layers(ly, start, end, 0);
    if (!ci.mixed) return;
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

}  // namespace aps

using namespace aps;

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
    const dim3 bgrid((unsigned)(od.ng > 1 ? od.ng - 1 : 1));  // one block per ring-segment boundary
#define APS_LAUNCH_X(v)                                                                                     \
    if (vm & (1u << (v))) {                                                                                 \
        if (acc == APS_ACC_KAHAN) {                                                                         \
            hipLaunchKernelGGL((k_sim_reduce_ex<v, true>), grid, dim3(BLOCK), 0, s, a, ly, pal, od);       \
            if (od.ng > 1)                                                                                  \
                hipLaunchKernelGGL((k_sim_reduce_ex_cross<v, true>), bgrid, dim3(BLOCK), 0, s, a, ly, pal, od); \
        } else {                                                                                            \
            hipLaunchKernelGGL((k_sim_reduce_ex<v, false>), grid, dim3(BLOCK), 0, s, a, ly, pal, od);      \
            if (od.ng > 1)                                                                                  \
                hipLaunchKernelGGL((k_sim_reduce_ex_cross<v, false>), bgrid, dim3(BLOCK), 0, s, a, ly, pal, od); \
        }                                                                                                   \
    }
    APS_FOR_VARIANTS(APS_LAUNCH_X)
#undef APS_LAUNCH_X
    if (fmt_idx && n_fmts > 1 && L > 1) {  // chunks that mix palette entries
        if (acc == APS_ACC_KAHAN)
            hipLaunchKernelGGL(k_sim_reduce_ex_slow<true>, dim3((unsigned)nchunks), dim3(BLOCK), 0, s, a, ly, pal, od);
        else
            hipLaunchKernelGGL(k_sim_reduce_ex_slow<false>, dim3((unsigned)nchunks), dim3(BLOCK), 0, s, a, ly, pal, od);
    }
    return launched();
}
