// aps_quant.hip -- scale and cast (Algorithm 1: the gradient times 2^ft,
// rounded to the custom format), and back to fp32 with the scale undone,
// with packed codes.
#include "aps_common.hpp"

namespace aps {

// ======================================================= K3: quantize

struct QuantArgs {
    const float* X;
    float* Q;  // may alias X: each element is read before its own store
    uint8_t* __restrict__ codes;
    int64_t ld;
    int32_t W;
    int32_t code_cls;
};

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


// Mixed-format chunks, all W rows; grid (boundary, row group): block y takes
// rows y, y + gridDim.y, ... (a grid's y extent is limited to 65535 blocks);
// element pairs per thread as in k_sim_reduce_mixed.
__global__ __launch_bounds__(BLOCK) void k_quantize_mixed(QuantArgs a, Layers ly, Pal pal) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    int64_t start, end;
    if (!mixed_chunk_of_boundary(ly, blockIdx.x, start, end)) return;
    for (int64_t w = blockIdx.y; w < a.W; w += gridDim.y) {
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
}

// Row blocks per boundary of k_quantize_mixed: one row per block up to this
// many workers, more rows per block beyond.
constexpr int32_t MIXED_ROW_BLOCKS = 4096;

// ===================================================== K5: dequantize

struct DeqArgs {
    const float* Q;  // may alias out
    const uint8_t* __restrict__ codes;
    float* out;
    int32_t code_cls;
};

// A thread's 4 elements of one chunk as loaded: the fp32 bit patterns, or
// the 4 codes (one 2-, 4- or 8-byte load, by code class).
struct DeqRaw {
    uint32_t w[4];
};

template <int IN>  // 0: fp32 values; 1 + code class: codes
__device__ __forceinline__ DeqRaw deq_load(const DeqArgs& a, int64_t j) {
    DeqRaw r;
    if constexpr (IN == 0) {
        const f4 v = __builtin_nontemporal_load((const f4*)(a.Q + j));
        r.w[0] = f2u(v.x);
        r.w[1] = f2u(v.y);
        r.w[2] = f2u(v.z);
        r.w[3] = f2u(v.w);
    } else if constexpr (IN == 1) {  // nibbles: elements j..j+3 in 2 bytes
        const uint32_t h = __builtin_nontemporal_load((const uint16_t*)(a.codes + (j >> 1)));
        r.w[0] = h & 15u;
        r.w[1] = (h >> 4) & 15u;
        r.w[2] = (h >> 8) & 15u;
        r.w[3] = h >> 12;
    } else if constexpr (IN == 2) {  // bytes
        const uint32_t b = __builtin_nontemporal_load((const uint32_t*)(a.codes + j));
        r.w[0] = b & 255u;
        r.w[1] = (b >> 8) & 255u;
        r.w[2] = (b >> 16) & 255u;
        r.w[3] = b >> 24;
    } else {  // little-endian uint16
        const u2v b = __builtin_nontemporal_load((const u2v*)(a.codes + 2 * j));
        r.w[0] = b.x & 0xFFFFu;
        r.w[1] = b.x >> 16;
        r.w[2] = b.y & 0xFFFFu;
        r.w[3] = b.y >> 16;
    }
    return r;
}

// Chunks a block has in flight at once: their loads are issued together, so
// each wave waits for memory once per DEQ_GROUP chunks (the work per chunk
// is 4 elements per thread, too little to cover a load's latency).
constexpr int DEQ_GROUP = 4;

// Codes of up to 8 bits decode through a table in LDS, one per palette
// entry (value of every code), filled once per block; 16-bit codes decode
// arithmetically.  A block walks its chunks in groups of DEQ_GROUP: the loads
// of the next group are issued before the current one is decoded and
// stored, and the first group's before the table is filled, so each wave
// has a group's loads in flight while it works.
template <int IN>
__global__ __launch_bounds__(BLOCK) void k_dequantize(DeqArgs a, Layers ly, Pal pal) {
    constexpr bool TABLE = IN == 1 || IN == 2;
    constexpr int NCODES = IN == 1 ? 16 : 256;
    __shared__ FmtK spal[APS_MAX_FORMATS];
    __shared__ float lut[TABLE ? APS_MAX_FORMATS : 1][TABLE ? NCODES : 1];
    auto setup = [&]() {
        pal_to_lds(pal, spal);
        if constexpr (TABLE) {
            for (int t = threadIdx.x; t < ly.n_fmts * NCODES; t += BLOCK)
                lut[t / NCODES][t % NCODES] = decode((uint32_t)(t % NCODES), spal[t / NCODES]);
            __syncthreads();
        }
    };
    auto dec = [&](uint32_t code, int p, const FmtK& f) -> float {
        if constexpr (TABLE) return lut[p][code];
        else return decode(code, f);
    };
    const int64_t nchunks = (ly.n + CH - 1) / CH;
    int64_t cb, ce;
    block_range(nchunks, cb, ce);
    // the group's loads are unconditional (a branch around each would make
    // the compiler wait for it before the next): past the block's last chunk
    // a thread loads that chunk again, past the gradient's end its last whole
    // group of 4, and ignores what it loaded
    const int64_t jlast = (ly.n & ~(int64_t)3) - 4;
    auto one = [&](int64_t jj, int li) {  // element jj of layer li, on its own
        const int p = ly.fmt_idx ? ly.fmt_idx[li] : 0;
        const int32_t ft = ly.scale_exp ? clamp_exp(ly.scale_exp[li]) : 0;
        const float v = IN == 0 ? a.Q[jj] : dec(load_code(a.codes, jj, a.code_cls), p, spal[p]);
        a.out[jj] = __builtin_amdgcn_ldexpf(v, -ft);
    };
    if (jlast < 0) {  // fewer than 4 elements: no whole group to load
        setup();
        if (blockIdx.x == 0 && threadIdx.x < ly.n) one(threadIdx.x, find_layer(ly.offsets, ly.L, threadIdx.x, 0));
        return;
    }
    if (cb >= ce) return;  // uniform per block
    int hint = 0;
    ChunkInfo cis[DEQ_GROUP];
    DeqRaw raw[DEQ_GROUP];
    // the chunks' layers first (scalar loads, wave-uniform), then the group's
    // data loads, all in flight together
    auto issue = [&](int64_t c0) {
        // usually the whole group lies in one layer: one lookup for all of it
        const int64_t gend = min(min(c0 + DEQ_GROUP, ce) * CH, ly.n);
        const ChunkInfo gi = chunk_layers(ly, c0 * CH, gend, hint);
        hint = __builtin_amdgcn_readfirstlane(gi.i0);
        if (gi.i0 == gi.i1) {
#pragma unroll
            for (int g = 0; g < DEQ_GROUP; ++g) cis[g] = gi;
        } else {
#pragma unroll
            for (int g = 0; g < DEQ_GROUP; ++g) {
                const int64_t c = min(c0 + g, ce - 1);
                cis[g] = chunk_layers(ly, c * CH, min(c * CH + CH, ly.n), hint);
                hint = __builtin_amdgcn_readfirstlane(cis[g].i0);
            }
        }
#pragma unroll
        for (int g = 0; g < DEQ_GROUP; ++g) {
            const int64_t j = min(c0 + g, ce - 1) * CH + (int64_t)threadIdx.x * VEC;
            raw[g] = deq_load<IN>(a, min(j, jlast));
        }
    };
    auto process = [&](int64_t c0, const ChunkInfo* gci, const DeqRaw* graw) {
#pragma unroll
        for (int g = 0; g < DEQ_GROUP; ++g) {
            const int64_t c = c0 + g;
            if (c >= ce) break;
            const int64_t start = c * CH;
            const int64_t end = min(start + CH, ly.n);
            const ChunkInfo& ci = gci[g];
            const int64_t j = start + (int64_t)threadIdx.x * VEC;
            if (j >= end) continue;
            if (ci.i0 == ci.i1 && j + 4 <= end) {
                // one layer: uniform format and exponent, 16-byte stores
                const FmtK& f = pal.f[ci.pidx];
                const int32_t ft = ly.scale_exp ? clamp_exp(cld(ly.scale_exp, ci.i0)) : 0;
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = IN == 0 ? u2f(graw[g].w[e]) : dec(graw[g].w[e], ci.pidx, f);
                const f4 o = {__builtin_amdgcn_ldexpf(v[0], -ft), __builtin_amdgcn_ldexpf(v[1], -ft),
                              __builtin_amdgcn_ldexpf(v[2], -ft), __builtin_amdgcn_ldexpf(v[3], -ft)};
                __builtin_nontemporal_store(o, (f4*)(a.out + j));  // out may alias Q: same elements
                continue;
            }
            // several layers in the chunk, or the gradient's ragged end: element by element
            int li = ci.i0;
            for (int e = 0; e < 4; ++e) {
                const int64_t jj = j + e;
                if (jj >= end) break;
                while (ly.offsets[li + 1] <= jj) ++li;
                one(jj, li);
            }
        }
    };
    issue(cb);
    setup();
    const int64_t ngroups = (ce - cb + DEQ_GROUP - 1) / DEQ_GROUP;
    for (int64_t k = 0; k + 1 < ngroups; ++k) {
        ChunkInfo cur_ci[DEQ_GROUP];
        DeqRaw cur[DEQ_GROUP];
#pragma unroll
        for (int g = 0; g < DEQ_GROUP; ++g) {
            cur_ci[g] = cis[g];
            cur[g] = raw[g];
        }
        issue(cb + (k + 1) * DEQ_GROUP);
        process(cb + k * DEQ_GROUP, cur_ci, cur);
    }
    process(cb + (ngroups - 1) * DEQ_GROUP, cis, raw);
}

}  // namespace aps

using namespace aps;

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
    // launch width measured on MI355X: with few rows per chunk (W < 64),
    // 64 blocks per CU (ResNet-50 at W = 8: 0.223 -> 0.20 ms)
    const dim3 grid((unsigned)grid_for(nchunks, W < 64 ? 64 : BLOCKS_PER_CU));
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
    APS_LAUNCH_Q(V_TOP_M0) APS_LAUNCH_Q(V_LOW_F64) APS_LAUNCH_Q(V_LOW_M0) APS_LAUNCH_Q(V_GEN)
#undef APS_LAUNCH_Q
    if (fmt_idx && n_fmts > 1 && L > 1)
        hipLaunchKernelGGL(k_quantize_mixed, dim3((unsigned)L, (unsigned)std::min<int32_t>(W, MIXED_ROW_BLOCKS)),
                           dim3(BLOCK), 0, s, a, ly, pal);
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
    // measured on MI355X (ResNet-50's 25.6 M byte codes, the next group's
    // loads issued before the current group is stored): 16 blocks per CU with
    // 4 chunks per group (30.7 us) beat 8 with 4 or 8, 16 with 2, 32 with 2
    // and 4 with 8 (31.6 to 35.5 us)
    const dim3 grid((unsigned)grid_for(nchunks, 16));
    hipStream_t s = (hipStream_t)stream;
    const int in = Q ? 0 : 1 + ccls;
    if (in == 0) hipLaunchKernelGGL(k_dequantize<0>, grid, dim3(BLOCK), 0, s, a, ly, pal);
    else if (in == 1) hipLaunchKernelGGL(k_dequantize<1>, grid, dim3(BLOCK), 0, s, a, ly, pal);
    else if (in == 2) hipLaunchKernelGGL(k_dequantize<2>, grid, dim3(BLOCK), 0, s, a, ly, pal);
    else hipLaunchKernelGGL(k_dequantize<3>, grid, dim3(BLOCK), 0, s, a, ly, pal);
    return launched();
}

// Instantiates only the product modes a variant can take: GP_FIT needs the
// TOP or LOW class with m >= 1; INT-class formats (k = 0) are always scaled.
