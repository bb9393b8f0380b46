// aps_sync.hip -- one whole APS synchronisation in one call (Algorithm 1 with
// the low-precision accumulator of Sec. 5), reading the W workers'
// gradients once where it can.
#include <atomic>
#include <mutex>

#include "aps_common.hpp"

namespace aps {

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
// whole chunk with the streaming kernel's row walk when many do.  With fewer
// than SYNC_BYTES_MIN_W workers only the per-256 minima are kept and whole
// 256-element groups are rerun; from SYNC_HALF_MIN_W workers on (m <= 7)
// the sums themselves are kept in 2 bytes and widened in the second pass.
// An accepted sum is a multiple of 2^(-126 - m) (T >= 2^-126), so its fp32
// pattern, normal or not, has no bits below position 23 - m >= 16.

// Zero the layer maxima before pass 1 accumulates them with atomicMax, and
// the repair list's length before pass 2 appends to it.
__global__ void k_sync_clear(uint32_t* __restrict__ maxabs, int32_t L, uint32_t* __restrict__ count) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < L) maxabs[i] = 0u;
    if (i == 0) *count = 0u;
}

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
    uint16_t* __restrict__ half;   // [round_up(n, CH)] top halves of the pass-1 sums, or null
    int32_t* __restrict__ guess;   // [L] guessed exponents (guessed-scale route)
    uint8_t* __restrict__ listed;  // [nchunks] 1 where the chunk is on the repair list
    bool bytes;                    // pass 1 stores minb for the single-entry chunks
};

// From this many workers on, and when every palette entry has m <= 7, pass 1
// writes each sum's top 16 bits instead of the fp32 value: the unscaled
// chain keeps m+1 significant bits, so the low 16 bits of its fp32 pattern
// are zero.  Pass 2 widens them into out (in k_sync_repair).  Writes in the
// middle of pass 1's row reads cost far more than their bytes at large W;
// the widening is one short streaming pass.  At small W the writes cost
// less and the widening more than it saves.
constexpr int32_t SYNC_HALF_MIN_W = 128;

// Fewer workers than this: pass 1 keeps only the per-wave minima, and pass 2
// reruns each 256-element group whose minimum is below its chunk's largest
// threshold.  Such a group is W rows of 1 KB, cheap to rerun at small W,
// while the per-element byte stores slow pass 1 down by more than their
// share of its traffic.
constexpr int32_t SYNC_BYTES_MIN_W = 64;

// What k_sync_repair does with a listed chunk.
enum RepairMode {
    RM_ELEMENTS = 0,  // find the flagged elements from their bytes
    RM_CHUNKS = 1,    // rerun all four quarters (guessed-scale route)
    RM_QUARTERS = 2,  // rerun the quarters whose wave minimum is below the chunk's threshold
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

// A thread's finished first-pass results for 4 elements, handed on (to its
// LDS slots below) after the next chunk's loads have been issued; lane 0 of
// a wave also holds the wave's minimum byte.
struct PendingSync {
    f4 o;
    uint32_t mb;  // the 4 exponent bytes, element j in the low byte
    uint32_t wb;  // wave minimum (lane 0)
    int64_t j, lim, c;
    bool valid;
};

// A thread's finished records wait in LDS (its own slots: no other thread
// reads them, so no barrier) and are written out STAGE chunks at a time, or
// when the block is done.  Writes in the middle of the row reads cost pass 1
// far more than their bytes; fewer, larger bursts of them cost less.
constexpr int STAGE = 8;

struct Stage {
    f4* o;         // [STAGE][BLOCK] sums
    uint32_t* mb;  // [STAGE][BLOCK] exponent bytes
    int32_t* j;    // [STAGE][BLOCK] first element (n <= 2^30)
    int cnt;       // this thread's filled slots
};

__device__ __forceinline__ void drain_stage(const SyncArgs& a, const SyncWs& ws, Stage& st, int64_t n) {
    const int t = threadIdx.x;
    for (int s = 0; s < st.cnt; ++s) {
        const int64_t j = st.j[s * BLOCK + t];
        const int64_t lim = min((j / CH) * CH + CH, n);
        const f4 o = st.o[s * BLOCK + t];
        if (ws.half) {
            // elements j, j+1 in the first word (low half first); the array is
            // padded to whole chunks, so all 8 bytes are in bounds
            const u2v h = {(f2u(o.x) >> 16) | (f2u(o.y) & 0xFFFF0000u), (f2u(o.z) >> 16) | (f2u(o.w) & 0xFFFF0000u)};
            __builtin_nontemporal_store(h, (u2v*)(ws.half + j));
        } else if (j + 4 <= lim) {
            __builtin_nontemporal_store(o, (f4*)(a.out + j));
        } else {
            if (j < lim) a.out[j] = o.x;
            if (j + 1 < lim) a.out[j + 1] = o.y;
            if (j + 2 < lim) a.out[j + 2] = o.z;
        }
        // the byte array is padded to whole chunks: a full word is always in bounds
        if (ws.bytes) __builtin_nontemporal_store(st.mb[s * BLOCK + t], (uint32_t*)(ws.minb + j));
    }
    st.cnt = 0;
}

__device__ __forceinline__ void flush_sync(const SyncArgs& a, const SyncWs& ws, PendingSync& pd, Stage& st,
                                           int64_t n) {
    if (!pd.valid) return;
    pd.valid = false;
    const int t = threadIdx.x;
    st.o[st.cnt * BLOCK + t] = pd.o;
    st.mb[st.cnt * BLOCK + t] = pd.mb;
    st.j[st.cnt * BLOCK + t] = (int32_t)pd.j;
    ++st.cnt;
    if ((threadIdx.x & 63) == 0) ws.wmin[pd.c * 4 + (threadIdx.x >> 6)] = (uint8_t)pd.wb;
    if (st.cnt == STAGE) drain_stage(a, ws, st, n);
}

// Pass 1 over the chunks of one palette entry (chunks that mix entries:
// k_sync_spec_mixed).  The format's rounding constants are uniform, so they
// sit in scalar registers.
__global__ __launch_bounds__(BLOCK) void k_sync_spec(SyncArgs a, SyncWs ws, Layers ly, Pal pal,
                                                    uint32_t* __restrict__ maxabs) {
    __shared__ uint32_t red[BLOCK / 64];
    __shared__ f4 st_o[STAGE * BLOCK];
    __shared__ uint32_t st_mb[STAGE * BLOCK];
    __shared__ int32_t st_j[STAGE * BLOCK];
    Stage st{st_o, st_mb, st_j, 0};
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
        if (ci.mixed) continue;  // k_sync_spec_mixed
        const int64_t j = start + (int64_t)threadIdx.x * VEC;
        uint32_t mx0 = 0, mx1 = 0, mx2 = 0, mx3 = 0;
        uint32_t tmin = 255u;  // this thread's smallest exponent byte
        if (j < end) {
            const FmtK& f = pal.f[ci.pidx];
            const uint32_t hf = f.half, sh = f.sh, lw = f.lsbw, mk = f.mask;
            const float sc = u2f((uint32_t)(124 - f.m) << 23);  // 2^-(m+3)
            uint32_t mn0, mn1, mn2, mn3;
            float s0, s1, s2, s3;
            const float* p = a.G + j;
            const int64_t ld = a.ld;
            stream_rows(
                a.W, [&](int r) { return ld4(p + (int64_t)r * ld); },
                [&]() { flush_sync(a, ws, pd, st, ly.n); },
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
                    s0 = u2f(rho(b0, hf, sh, lw, mk));
                    s1 = u2f(rho(b1, hf, sh, lw, mk));
                    s2 = u2f(rho(b2, hf, sh, lw, mk));
                    s3 = u2f(rho(b3, hf, sh, lw, mk));
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
                    mn0 = min(mn0, max(a0 - 1u, f2u(u2f(f2u(s0) & 0x7FFFFFFFu) * sc)));
                    mn1 = min(mn1, max(a1 - 1u, f2u(u2f(f2u(s1) & 0x7FFFFFFFu) * sc)));
                    mn2 = min(mn2, max(a2 - 1u, f2u(u2f(f2u(s2) & 0x7FFFFFFFu) * sc)));
                    mn3 = min(mn3, max(a3 - 1u, f2u(u2f(f2u(s3) & 0x7FFFFFFFu) * sc)));
                    s0 = u2f(rho(f2u(s0 + u2f(rho(b0, hf, sh, lw, mk))), hf, sh, lw, mk));
                    s1 = u2f(rho(f2u(s1 + u2f(rho(b1, hf, sh, lw, mk))), hf, sh, lw, mk));
                    s2 = u2f(rho(f2u(s2 + u2f(rho(b2, hf, sh, lw, mk))), hf, sh, lw, mk));
                    s3 = u2f(rho(f2u(s3 + u2f(rho(b3, hf, sh, lw, mk))), hf, sh, lw, mk));
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
        // every lane of the wave takes part in the minimum; lane 0 has the
        // wave's first element, so it holds this chunk's record whenever the
        // wave has one.  A lane without an element here keeps the record of
        // an earlier chunk, whose minimum must stay as it is.
        const uint32_t wmin_here = wave_min_u32(tmin);
        if (j < end) pd.wb = wmin_here;
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
    flush_sync(a, ws, pd, st, ly.n);
    drain_stage(a, ws, st, ly.n);
}

// Pass 1 over the chunks that mix palette entries, one block per layer
// boundary (the block of the first boundary inside a chunk owns it), one
// element per thread: the same chain, maximum and byte as k_sync_spec.  The
// scan skips these chunks; k_sync_repair_mixed reads their bytes.
__global__ __launch_bounds__(BLOCK) void k_sync_spec_mixed(SyncArgs a, SyncWs ws, Layers ly, Pal pal,
                                                          uint32_t* __restrict__ maxabs) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    int64_t start, end;
    if (!mixed_chunk_of_boundary(ly, blockIdx.x, start, end)) return;
    for (int64_t j = start + threadIdx.x; j < end; j += BLOCK) {
        const int li = find_layer(ly.offsets, ly.L, j, 0);
        const FmtK& f = spal[ly.fmt_idx[li]];
        const float sc = u2f((uint32_t)(124 - f.m) << 23);  // 2^-(m+3)
        const float* p = a.G + j;
        uint32_t b = f2u(p[0]);
        uint32_t mx = b & 0x7FFFFFFFu;
        uint32_t mn = mx - 1u;  // a zero wraps to the top and never wins the min
        float s = u2f(rho(b, f.half, f.sh, f.lsbw, f.mask));
        for (int w = 1; w < a.W; ++w) {
            b = f2u(p[(int64_t)w * a.ld]);
            const uint32_t ab = b & 0x7FFFFFFFu;
            mx = max(mx, ab);
            mn = min(mn, max(ab - 1u, f2u(u2f(f2u(s) & 0x7FFFFFFFu) * sc)));
            s = u2f(rho(f2u(s + u2f(rho(b, f.half, f.sh, f.lsbw, f.mask))), f.half, f.sh, f.lsbw, f.mask));
        }
        if (ws.half)
            ws.half[j] = (uint16_t)(f2u(s) >> 16);
        else
            a.out[j] = s;
        ws.minb[j] = (uint8_t)min(mn >> 23, 255u);
        if (mx) atomicMax(maxabs + li, mx);
    }
}

// A layer's scale exponent (as k_scales) and its repair threshold: an
// element is recomputed when its exponent byte is below th.  th = 256
// recomputes the whole layer (ghat INF/NaN, N * ghat = INF or above 2^127);
// an all-zero layer needs nothing (0).
__device__ __forceinline__ void sync_layer(uint32_t maxabs_bits, int32_t N, const FmtK& f, int32_t& r, int32_t& th) {
    const uint32_t gb = maxabs_bits & 0x7FFFFFFFu;
    r = 0;
    th = 256;
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
}

// Pass 2's bookkeeping in one launch; thread t handles layer t and chunk t.
//  * Layer t: its exponent into scale_exp and its threshold into thr (the
//    one-pass route), or the exponent and a mark in thr, 1 where the guess
//    in ws.guess differed (the guessed-scale route).
//  * Chunk t (single palette entry): listed for repair when its minimum
//    byte is below the largest threshold among its layers (one-pass: never
//    misses a flagged element; the repair looks at each), or when one of its
//    layers was guessed wrong (guessed scales).  The chunk's thresholds are
//    recomputed here from the maxima, not read from thr, which other threads
//    of this launch are writing.  The list's length was zeroed in pass 1.
__global__ void k_sync_bookkeep(const uint32_t* __restrict__ maxabs, Layers ly, int32_t N, Pal pal,
                                int32_t* __restrict__ scale_exp, SyncWs ws, bool guess) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    // what decides a layer's repair: its threshold, or whether its guess was wrong
    auto layer_th = [&](int i, int32_t& r) {
        const FmtK& f = spal[ly.fmt_idx ? ly.fmt_idx[i] : 0];
        int32_t th;
        sync_layer(maxabs[i], N, f, r, th);
        return guess ? (clamp_exp(r) != clamp_exp(ws.guess[i]) ? 1 : 0) : th;
    };
    if (t < ly.L) {
        int32_t r;
        const int32_t th = layer_th((int)t, r);
        scale_exp[t] = r;
        ws.thr[t] = th;
    }
    const int64_t nchunks = (ly.n + CH - 1) / CH;
    if (t >= nchunks) return;
    const int64_t start = t * CH;
    const int64_t end = min(start + CH, ly.n);
    uint32_t cm = 0u;  // the guessed-scale route reruns whole chunks: every element counts as byte 0
    if (!guess) {
        const uint32_t w4 = *(const uint32_t*)(ws.wmin + 4 * t);
        cm = 255u;
        for (int wv = 0; wv < 4; ++wv)
            if (start + 256 * wv < end) cm = min(cm, (w4 >> (8 * wv)) & 0xFFu);
    }
    const int i0 = find_layer(ly.offsets, ly.L, start, 0), i1 = find_layer(ly.offsets, ly.L, end - 1, i0);
    int32_t th = 0;
    bool mixed = false;
    const int p0 = ly.fmt_idx ? ly.fmt_idx[i0] : 0;
    for (int i = i0; i <= i1; ++i) {
        if (ly.offsets[i] == ly.offsets[i + 1]) continue;  // empty layer
        int32_t r;
        th = max(th, layer_th(i, r));
        if (ly.fmt_idx && ly.fmt_idx[i] != p0) mixed = true;
    }
    const bool listed = !mixed && (int32_t)cm < th;
    if (listed) ws.list[atomicAdd(ws.count, 1u)] = (int32_t)t;
    ws.listed[t] = listed ? 1 : 0;
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

// One wave widens a chunk's pass-1 sums, kept as top halves, into out: four
// steps of 4 elements per lane, so that each step's loads (8 bytes per lane)
// and stores (16) are contiguous across the wave.  The half array is padded
// to whole chunks.
__device__ __forceinline__ void widen_chunk(const SyncWs& ws, float* __restrict__ out, int64_t start, int64_t n) {
    const int lane = threadIdx.x & 63;
    u2v h[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) h[q] = __builtin_nontemporal_load((const u2v*)(ws.half + start + 256 * q + 4 * lane));
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int64_t j = start + 256 * q + 4 * lane;
        const f4 v = {u2f(h[q].x << 16), u2f(h[q].x & 0xFFFF0000u), u2f(h[q].y << 16), u2f(h[q].y & 0xFFFF0000u)};
        if (j + 4 <= n) {
            __builtin_nontemporal_store(v, (f4*)(out + j));
        } else {
            for (int e = 0; e < 4 && j + e < n; ++e) out[j + e] = v[e];
        }
    }
}

// Second pass over the listed chunks of one variant's format, one wave per
// chunk: find the flagged elements (16 bytes per lane), then repair them one
// after another (at most SPARSE_MAX), or rerun the whole chunk through the
// streaming row walk, a quarter at a time.  Waves stride over the list; its
// length is read on the device.  Without bytes (RM_CHUNKS, RM_QUARTERS) a
// listed chunk's four quarters are four tasks, so few listed chunks still
// spread over many waves; RM_QUARTERS skips a quarter whose wave minimum is
// not below the largest threshold of the chunk's layers (no element of it
// can be flagged).
// Halves are kept only on the one-pass route with bytes (RM_ELEMENTS), where
// each listed chunk has one wave: it widens the chunk, then repairs it.
template <int V>
__global__ __launch_bounds__(BLOCK) void k_sync_repair(ReduceArgs a, Layers ly, Pal pal, SyncWs ws, int mode,
                                                      bool widen_rest) {
    const bool every = mode != RM_ELEMENTS;
    const int64_t total = (int64_t)*ws.count * (every ? 4 : 1);
    const int lane = threadIdx.x & 63;
    const int64_t nw = (int64_t)gridDim.x * (BLOCK / 64);
    const int64_t wave = __builtin_amdgcn_readfirstlane((int)(blockIdx.x * (BLOCK / 64) + (threadIdx.x >> 6)));
    if (ws.half && widen_rest) {
        // the sums kept as halves (pass 1 from SYNC_HALF_MIN_W workers on):
        // one launch widens every chunk that is not listed, mixed ones
        // included (k_sync_repair_mixed runs after it); a listed chunk is
        // widened by the wave that repairs it, just before its repairs
        const int64_t nchunks = (ly.n + CH - 1) / CH;
        for (int64_t c = wave; c < nchunks; c += nw)
            if (!ws.listed[c]) widen_chunk(ws, a.out, c * CH, ly.n);
    }
    for (int64_t k = wave; k < total; k += nw) {
        const int64_t start = (int64_t)cld(ws.list, every ? k >> 2 : k) * CH;
        const int64_t end = min(start + CH, ly.n);
        const ChunkInfo ci = chunk_layers(ly, start, end, 0);
        const FmtK& f = pal.f[ci.pidx];
        if (f.variant != V) continue;  // another launch owns this format
        if (ws.half) {
            widen_chunk(ws, a.out, start, ly.n);
            __threadfence_block();  // the widened values are stored before any repair of the chunk
        }
        // 16 consecutive elements per lane; the byte array is padded to whole chunks
        const int64_t j0 = start + 16 * lane;
        uint32_t mask = 0;
        if (every) {
            mask = ~0u;  // more than SPARSE_MAX: the whole chunk below
        } else if (ci.i0 == ci.i1) {  // one layer: one threshold, read once
            const u4v w = *(const u4v*)(ws.minb + j0);
            const int32_t th = cld(ws.thr, ci.i0);
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const uint32_t byte = (w[e >> 2] >> (8 * (e & 3))) & 0xFFu;
                if ((int32_t)byte < th && j0 + e < end) mask |= 1u << e;
            }
        } else {
            const u4v w = *(const u4v*)(ws.minb + j0);
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
            const int q0 = every ? (int)(k & 3) : 0, q1 = every ? q0 + 1 : 4;
            if (mode == RM_QUARTERS) {
                int32_t th = 0;
                for (int li = ci.i0; li <= ci.i1; ++li) th = max(th, cld(ws.thr, li));
                if ((int32_t)ws.wmin[(start / CH) * 4 + q0] >= th) continue;
            }
#pragma unroll 1
            for (int qtr = q0; qtr < q1; ++qtr) {
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

// Flagged elements of chunks that mix palette entries, element by element
// (with every: all of their elements).
__global__ __launch_bounds__(BLOCK) void k_sync_repair_mixed(ReduceArgs a, Layers ly, Pal pal, SyncWs ws,
                                                            bool every) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    int64_t start, end;
    if (!mixed_chunk_of_boundary(ly, blockIdx.x, start, end)) return;
    for (int64_t j = start + threadIdx.x; j < end; j += BLOCK) {
        const int li = find_layer(ly.offsets, ly.L, j, 0);
        if (!every && (int32_t)ws.minb[j] >= ws.thr[li]) continue;
        const FmtK& f = spal[ly.fmt_idx[li]];
        const int F = clamp_exp(ly.scale_exp[li]) + f.k;
        a.out[j] = __builtin_amdgcn_ldexpf(reduce_elem_any(a, f, j, F), -F);
    }
}

// ======================================= K5b: the guessed-scale route
//
// For a format of narrow range at large W most elements have an input in
// the scaled subnormal range, and the one-pass route would recompute nearly
// all of them.  There pass 1 runs the scaled path itself, with a guessed
// exponent per layer, and takes the true maxima alongside.  Wherever the
// guess equals the exponent the maxima give, pass 1 did exactly the scaled
// path's arithmetic; pass 2 reruns every chunk of a layer whose guess was
// wrong.  The guess comes from the maxima of every GUESS_ROW_STRIDE-th
// worker (a sample of n_s values of a layer, K = W / rows times fewer than
// the layer has).  The max over all workers is larger than the sample's: for
// normal values the max of n draws grows like sqrt(2 ln n), so by about
// sqrt(1 + ln K / ln n_s).  The guess takes the sample's fl32(N * max) times
// that factor.  It affects only how much pass 2 reruns, never a result.

constexpr int GUESS_ROW_STRIDE = 32;

// The guessed exponent of each layer from the sampled maxima (rows sampled
// rows of N), into guess: as k_scales, on the sample's N * max raised by the
// expected growth of the max.  Also zeroes the repair list's length.
__global__ void k_guess_scales(const uint32_t* __restrict__ maxabs, Layers ly, int32_t N, int32_t rows, Pal pal,
                               int32_t* __restrict__ guess, uint32_t* __restrict__ count) {
    __shared__ FmtK spal[APS_MAX_FORMATS];
    pal_to_lds(pal, spal);
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0) *count = 0u;
    if (i >= ly.L) return;
    const FmtK& f = spal[ly.fmt_idx ? ly.fmt_idx[i] : 0];
    const uint32_t gb = maxabs[i] & 0x7FFFFFFFu;
    int32_t r = 0;
    if (gb != 0 && gb < 0x7F800000u) {
        const float t = (float)N * u2f(gb);
        uint32_t tb = f2u(t);
        if (tb < 0x7F800000u) {
            const float ns = (float)(ly.offsets[i + 1] - ly.offsets[i]) * (float)rows;
            const float grow = sqrtf(1.0f + logf((float)N / (float)rows) / logf(fmaxf(ns, 2.0f)));
            const uint32_t tn = f2u(t * grow);
            if (tn < 0x7F800000u) tb = tn;
            r = f.emax - ceil_log2_bits(tb);
        }
    }
    guess[i] = r;
}

// Pass 1 of the guessed-scale route over the chunks of one variant's format:
// the fused scaled sum of k_sim_reduce with the guessed exponents, plus the
// layer maxima (chunks that mix palette entries: maxima by
// k_sync_spec_mixed, sums in pass 2).
template <int V>
__global__ __launch_bounds__(BLOCK) void k_guess_spec(ReduceArgs a, Layers ly, Pal pal,
                                                     uint32_t* __restrict__ maxabs) {
    __shared__ uint32_t red[BLOCK / 64];
    const int64_t nchunks = (ly.n + CH - 1) / CH;
    int64_t cb, ce;
    block_range(nchunks, cb, ce);
    int hint = 0;
    uint32_t run = 0;  // running max of layer run_layer (chunks inside one layer)
    int run_layer = -1;
    PendingOut pd;
    pd.valid = false;
    for (int64_t c = cb; c < ce; ++c) {
        const int64_t start = c * CH;
        const int64_t end = min(start + CH, ly.n);
        const ChunkInfo ci = chunk_layers(ly, start, end, hint);
        hint = ci.i0;
        if (ci.mixed) continue;
        const FmtK& f = pal.f[ci.pidx];
        if (f.variant != V) continue;  // another launch owns this format
        const int64_t j = start + (int64_t)threadIdx.x * VEC;
        uint32_t mx[4] = {0u, 0u, 0u, 0u};
        if (j < end) {
            int32_t ft[4];
            if (ci.i0 == ci.i1) {
                const int32_t t = clamp_exp(cld(ly.scale_exp, ci.i0));
                ft[0] = ft[1] = ft[2] = ft[3] = t;
            } else {
                elem_scales(ly, ci, j, ft);
            }
            reduce_vec<V, true>(a, f, j, end, ft, pd, mx);
            // elements past the end of the gradient (row padding) do not count
            if (j + 1 >= end) mx[1] = 0;
            if (j + 2 >= end) mx[2] = 0;
            if (j + 3 >= end) mx[3] = 0;
        }
        if (ci.i0 == ci.i1) {
            const uint32_t v = max(max(mx[0], mx[1]), max(mx[2], mx[3]));
            if (ci.i0 != run_layer) {
                if (run_layer >= 0) block_max_atomic(run, maxabs + run_layer, red);
                run_layer = ci.i0;
                run = 0;
            }
            run = max(run, v);
        } else {
            for (int li = ci.i0; li <= ci.i1; ++li) {
                const int64_t lo = cld(ly.offsets, li), hi = cld(ly.offsets, li + 1);
                uint32_t v = 0;
                if (j < end)
                    for (int e = 0; e < 4; ++e)
                        if (j + e >= lo && j + e < hi) v = max(v, mx[e]);
                block_max_atomic(v, maxabs + li, red);
            }
        }
    }
    if (run_layer >= 0) block_max_atomic(run, maxabs + run_layer, red);
    flush_out(a, pd);
}

}  // namespace aps

using namespace aps;

// Workspace of aps_sync, in 256-byte aligned parts: the per-element exponent
// bytes (padded to whole chunks), four bytes per chunk, the int32 layer
// thresholds, the list counter, the int32 chunk list, two bytes per element
// (padded to whole chunks) for the top halves of the pass-1 sums, the int32
// guessed exponents.
struct SyncLayout {
    uint64_t minb, wmin, thr, count, list, half, guess, listed, total;
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
    o.half = o.list + up256(4u * nch);
    o.guess = o.half + up256(2u * nch * (uint64_t)CH);
    o.listed = o.guess + up256(4u * (uint64_t)L);
    o.total = o.listed + up256(nch);
    return o;
}

extern "C" uint64_t aps_sync_workspace_bytes(int64_t n, int32_t L) {
    if (n < 0 || L < 0 || n > APS_MAX_ELEMS) return 0;
    return sync_layout(n, L).total;
}

// Which route aps_sync takes.  The one-pass route applies when N = W is a
// power of two (exact N * ghat, no overflow) and every format has m <= 10
// (an fp32 add then one rounding equals rounding the exact sum) and rounds
// in fp32 (not class GEN: its subnormal grid reaches below 2^-126).  Without a
// route flag it is taken when it is also expected to pay: for layers of
// normally distributed values (max about 5 sigma) the threshold sits at
// W * 2^(emin - emax) of the layer's max, each input falls below it with
// probability about W * 2^(emin - emax + 2), and an element is recomputed
// with probability up to W^2 * 2^(emin - emax + 2); above 2^-7 most chunks
// would be recomputed.  Then the guessed-scale route is taken for sets of
// at least GUESS_MIN_WORK element-workers (its sample and extra launches
// cost more than they save on smaller ones), else two passes.
constexpr int64_t GUESS_MIN_WORK = (int64_t)1 << 26;

static bool one_pass_applies(int32_t W, const Pal& pal, int32_t n_fmts) {
    if (W & (W - 1)) return false;
    for (int i = 0; i < n_fmts; ++i)
        if (pal.f[i].m > 10 || pal.f[i].variant == V_GEN) return false;
    return true;
}

static int sync_route(int32_t W, int64_t n, const Pal& pal, int32_t n_fmts, uint32_t flags) {
    if (flags & APS_SYNC_TWO_PASS) return APS_SYNC_ROUTE_TWO_PASS;
    if (flags & APS_SYNC_GUESS) return APS_SYNC_ROUTE_GUESS;
    const bool applies = one_pass_applies(W, pal, n_fmts);
    if (flags & APS_SYNC_ONE_PASS) return applies ? APS_SYNC_ROUTE_ONE_PASS : APS_SYNC_ROUTE_TWO_PASS;
    bool pays = applies;
    int lw = 0;
    while ((1 << lw) < W) ++lw;
    for (int i = 0; i < n_fmts; ++i)
        if (2 * lw + pal.f[i].emin - pal.f[i].emax + 2 > -7) pays = false;
    if (pays) return APS_SYNC_ROUTE_ONE_PASS;
    return (int64_t)W * n >= GUESS_MIN_WORK ? APS_SYNC_ROUTE_GUESS : APS_SYNC_ROUTE_TWO_PASS;
}

static constexpr uint32_t ROUTE_BITS = APS_SYNC_ONE_PASS | APS_SYNC_TWO_PASS | APS_SYNC_GUESS;

static bool route_bits_ok(uint32_t flags) {
    const uint32_t r = flags & ROUTE_BITS;
    return (r & (r - 1)) == 0;  // at most one
}

extern "C" int aps_sync_route(int32_t W, int64_t n, const aps_format* fmts, int32_t n_fmts, uint32_t flags) {
    if (W < 1 || W > APS_MAX_WORKERS || n < 0 || n > APS_MAX_ELEMS) return APS_ERR_SIZE;
    if (!route_bits_ok(flags)) return APS_ERR_UNSUPPORTED;
    Pal pal;
    const int st = check_palette(fmts, n_fmts, pal, nullptr);
    if (st != APS_OK) return st;
    return sync_route(W, n, pal, n_fmts, flags);
}

extern "C" int aps_sync(const float* G, int32_t W, int64_t ld, int64_t n, const int64_t* offsets, int32_t L,
                        const aps_format* fmts, int32_t n_fmts, const uint8_t* fmt_idx, uint32_t flags,
                        uint32_t* maxabs_bits, int32_t* scale_exp, float* out, void* workspace,
                        uint64_t workspace_bytes, void* stream) {
    int st = check_rows(G, W, ld, n, offsets, L);
    if (st != APS_OK) return st;
    if (!maxabs_bits || !scale_exp || !workspace || (!out && n > 0)) return APS_ERR_NULL;
    const uint32_t phases = flags & (APS_SYNC_PASS1 | APS_SYNC_PASS2);
    if (phases == 0 || (flags & ~(APS_SYNC_PASS1 | APS_SYNC_PASS2 | ROUTE_BITS)) || !route_bits_ok(flags))
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
              (int32_t*)(wb + lay.list), nullptr, (int32_t*)(wb + lay.guess), wb + lay.listed, W >= SYNC_BYTES_MIN_W};
    Layers ly{offsets, fmt_idx, scale_exp, n, L, n_fmts};
    const int route = sync_route(W, n, pal, n_fmts, flags);
    if (route == APS_SYNC_ROUTE_ONE_PASS && W >= SYNC_HALF_MIN_W) {
        bool narrow = true;
        for (int i = 0; i < n_fmts; ++i) narrow = narrow && pal.f[i].m <= 7;
        if (narrow) ws.half = (uint16_t*)(wb + lay.half);
    }
    if (route == APS_SYNC_ROUTE_TWO_PASS) {
        // two passes: exactly the three calls of the step
        if (phases & APS_SYNC_PASS1) {
            st = aps_layer_maxabs(G, W, ld, n, offsets, L, maxabs_bits, stream);
            if (st != APS_OK) return st;
        }
        if (phases & APS_SYNC_PASS2) {
            st = aps_layer_scales(maxabs_bits, L, W, fmts, n_fmts, fmt_idx, scale_exp, stream);
            if (st != APS_OK) return st;
            st = aps_sim_reduce(G, W, ld, n, offsets, L, scale_exp, fmts, n_fmts, fmt_idx, 0u, out, nullptr, stream);
            if (st != APS_OK) return st;
        }
        return APS_OK;
    }
    const dim3 lgrid((unsigned)((L + 255) / 256));
    const bool mixed = fmt_idx && n_fmts > 1 && L > 1;
    const unsigned vm = variant_mask(pal, n_fmts);
    const dim3 grid((unsigned)stream_grid(nchunks, W, BLOCKS_PER_CU));  // pass-1 row walks
    // repairs: the list's length is only known on the device.  The one-pass
    // route is taken where few elements need recomputing (often none), so a
    // narrow grid, whose launch costs less; the guessed-scale route reruns
    // whole layers, a quarter chunk per wave.
    const bool guess = route == APS_SYNC_ROUTE_GUESS;
    const dim3 rgrid((unsigned)grid_for(nchunks, (guess || ws.half) ? BLOCKS_PER_CU : 4));
    ReduceArgs ra{G, out, nullptr, ld, W, 0u, 0};
    SyncArgs sa{G, out, ld, W};
    const int rmode = guess ? RM_CHUNKS : (ws.bytes ? RM_ELEMENTS : RM_QUARTERS);
    if (guess && (phases & APS_SYNC_PASS1)) {
        // the maxima of every GUESS_ROW_STRIDE-th worker give the guesses
        const int32_t rows = (W + GUESS_ROW_STRIDE - 1) / GUESS_ROW_STRIDE;
        st = aps_layer_maxabs(G, rows, rows > 1 ? ld * GUESS_ROW_STRIDE : ld, n, offsets, L, maxabs_bits, stream);
        if (st != APS_OK) return st;
        hipLaunchKernelGGL(k_guess_scales, lgrid, dim3(256), 0, s, maxabs_bits, ly, W, rows, pal, ws.guess, ws.count);
        if (n > 0) {
            // the full maxima accumulate on top of the sampled ones; the sums
            // take the guessed exponents
            Layers lg = ly;
            lg.scale_exp = ws.guess;
#define APS_LAUNCH_G(v) \
    if (vm & (1u << (v))) hipLaunchKernelGGL(k_guess_spec<v>, grid, dim3(BLOCK), 0, s, ra, lg, pal, maxabs_bits);
            APS_FOR_VARIANTS(APS_LAUNCH_G)
#undef APS_LAUNCH_G
            if (mixed)
                hipLaunchKernelGGL(k_sync_spec_mixed, dim3((unsigned)L), dim3(BLOCK), 0, s, sa, ws, ly, pal, maxabs_bits);
        }
    }
    if (!guess && (phases & APS_SYNC_PASS1)) {
        hipLaunchKernelGGL(k_sync_clear, lgrid, dim3(256), 0, s, maxabs_bits, L, ws.count);
        if (n > 0) {
            // launch width measured on MI355X: 24 blocks per CU for many rows,
            // 32 for few (shorter work per chunk), wider on large sets
            hipLaunchKernelGGL(k_sync_spec, dim3((unsigned)stream_grid(nchunks, W, W >= 64 ? 24 : 32)), dim3(BLOCK), 0,
                               s, sa, ws, ly, pal, maxabs_bits);
            if (mixed)
                hipLaunchKernelGGL(k_sync_spec_mixed, dim3((unsigned)L), dim3(BLOCK), 0, s, sa, ws, ly, pal, maxabs_bits);
        }
    }
    if (phases & APS_SYNC_PASS2) {
        const int64_t items = std::max<int64_t>(L, nchunks);
        hipLaunchKernelGGL(k_sync_bookkeep, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, s, maxabs_bits, ly, W,
                           pal, scale_exp, ws, guess);
        if (n > 0) {
            // the first repair launch also widens the sums kept as halves
            bool first = true;
#define APS_LAUNCH_S(v)                                                                                  \
    if (vm & (1u << (v))) {                                                                              \
        hipLaunchKernelGGL(k_sync_repair<v>, rgrid, dim3(BLOCK), 0, s, ra, ly, pal, ws, rmode, first); \
        first = false;                                                                                   \
    }
            APS_FOR_VARIANTS(APS_LAUNCH_S)
#undef APS_LAUNCH_S
            if (mixed)
                hipLaunchKernelGGL(k_sync_repair_mixed, dim3((unsigned)L), dim3(BLOCK), 0, s, ra, ly, pal, ws, guess);
        }
    }
    return launched();
}

// ================================= aps_sync without a caller's workspace
//
// The workspace of aps_sync_noalloc: one static array per GPU, placed there by
// the HIP runtime when it loads this code object on the device.  In host code
// `scratch` names the host-side shadow of the symbol, not device memory, so
// it is never passed to a kernel or a copy: the device address comes from
// hipGetSymbolAddress, taken once per device with that device current and
// kept in scratch_ptr.
static __device__ __align__(256) uint8_t scratch[APS_SYNC_SCRATCH_BYTES];

namespace {
constexpr int SCRATCH_MAX_DEVICES = 64;
std::atomic<void*> scratch_ptr[SCRATCH_MAX_DEVICES];
std::mutex scratch_mu;

// Device address of the current device's scratch array (APS_ERR_DEVICE if
// the runtime cannot give it).
int scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= SCRATCH_MAX_DEVICES) return APS_ERR_DEVICE;
    void* p = scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(scratch_mu);
        p = scratch_ptr[dev].load(std::memory_order_relaxed);
        if (!p) {
            if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return APS_ERR_DEVICE;
            if ((uintptr_t)p & 255u) return APS_ERR_DEVICE;
            scratch_ptr[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return APS_OK;
}
}  // namespace

extern "C" int aps_sync_noalloc(const float* G, int32_t W, int64_t ld, int64_t n, const int64_t* offsets,
                                int32_t L, const aps_format* fmts, int32_t n_fmts, const uint8_t* fmt_idx,
                                uint32_t flags, uint32_t* maxabs_bits, int32_t* scale_exp, float* out,
                                void* stream) {
    // the checks aps_sync makes on these arguments come first, so that a bad
    // call reports the same status; then the size against the array, all
    // before the device is touched
    int st = check_rows(G, W, ld, n, offsets, L);
    if (st != APS_OK) return st;
    if (!maxabs_bits || !scale_exp || (!out && n > 0)) return APS_ERR_NULL;
    if (sync_layout(n, L).total > APS_SYNC_SCRATCH_BYTES) return APS_ERR_SIZE;
    void* ws = nullptr;
    st = scratch_address(&ws);
    if (st != APS_OK) return st;
    return aps_sync(G, W, ld, n, offsets, L, fmts, n_fmts, fmt_idx, flags, maxabs_bits, scale_exp, out, ws,
                    APS_SYNC_SCRATCH_BYTES, stream);
}
