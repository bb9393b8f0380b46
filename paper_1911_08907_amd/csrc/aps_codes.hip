// aps_codes.hip -- the W-worker rounded sum over packed codes, the form in
// which workers would exchange the cast gradients (Algorithm 1's SUM
// all-reduce of the cast gradients; Sec. 5).
#include "aps_common.hpp"

namespace aps {

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
    // each wave's fp32 outputs pass through its own LDS slots, so that they
    // leave in stores of consecutive 16-byte pieces per lane (a lane's EPT
    // outputs written as EPT/4 stores 4*EPT bytes apart wrote up to 1.7x
    // the output's bytes to HBM)
    __shared__ __align__(16) float ostage[BLOCK * EPT];
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
        const int lane = threadIdx.x & 63;
        const int64_t wbase = j - (int64_t)lane * EPT;  // the wave's first element
        if (wbase + 64 * EPT <= end) {
            // the whole wave is inside the gradient: every lane is here
            if (a.out) {
                float* wbuf = ostage + (threadIdx.x - lane) * EPT;
#pragma unroll
                for (int q = 0; q < EPT / 4; ++q) {
                    const f4 v = {o[4 * q], o[4 * q + 1], o[4 * q + 2], o[4 * q + 3]};
                    *(f4*)(wbuf + lane * EPT + 4 * q) = v;
                }
                __builtin_amdgcn_wave_barrier();
#pragma unroll
                for (int q = 0; q < EPT / 4; ++q) {
                    const f4 v = *(const f4*)(wbuf + 4 * lane + 256 * q);
                    __builtin_nontemporal_store(v, (f4*)(a.out + wbase + 4 * lane + 256 * q));
                }
                __builtin_amdgcn_wave_barrier();
            }
            if (a.codes_out) {
                const u4v v = {cw[0], cw[1], cw[2], cw[3]};
                __builtin_nontemporal_store(v, (u4v*)(a.codes_out + code_byte(j, CC)));
            }
        } else {
            // the wave reaches the ragged end of the gradient: element by element
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
        case V_GEN: return reduce_codes_elem<V_GEN>(a, f, cc, j);
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

}  // namespace aps

using namespace aps;

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
