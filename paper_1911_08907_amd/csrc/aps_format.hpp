// aps_format.hpp -- custom-float constants and device rounding for gfx950.
//
// The cast to a custom float of Algorithm 1 (arXiv 1911.08907), with the
// round-to-nearest-even mode of Sec. 4, the format layout that reproduces
// Table 2, and the low-precision accumulator of Sec. 5.
//
// Working domain.  Every kernel rounds in a shifted copy of the format: a
// native value v is carried as v * 2^k with k = 127 - emax, so that the
// format's overflow threshold coincides with fp32's.  Power-of-two scaling is
// exact (Sec. 3.3.1), so rounding in the shifted domain and shifting back
// gives the same result as rounding natively, as long as nothing below the
// format's half-smallest-subnormal is decided by fp32's own underflow: the
// scaled input is an fp32 value, fl32(x * 2^ft), which fp32 itself has
// already rounded once it lies below 2^-126.  For e = 8 with bias 127 the
// shift is k = 0.  Formats for which that does not hold (e = 8 with another
// bias, or a half-smallest-subnormal below 2^-126) take class GEN below.
// In that domain:
//   * a value with |y| >= 2^emin (format normal range) is rounded on its
//     fp32 bit pattern: add half an ulp of the m-bit mantissa (plus the
//     lowest kept bit, for ties to even) and clear the dropped bits.  A carry
//     out of the mantissa bumps the exponent; at the top it produces the
//     bit pattern of INF, which is the format's overflow;
//   * a value below 2^emin (format subnormal range) is rounded onto the fixed
//     subnormal grid with one fp32 add/subtract of c0 = 2^(emin - m + 23)
//     ("magic" constant): fp32's own round-to-nearest-even does the work.
//     When c0 would not be an fp32 value (small e, class LOW), the value is
//     instead scaled so that the grid's step is 1 and rounded to an integer
//     (rint, ties to even), then scaled back: the step 2^(emin - m) lies
//     between 2^105 and 2^126 there, so both scalings are exact wherever the
//     result is not zero (m = 0 formats keep the add/subtract in a domain
//     shifted down by j more bits);
//   * for e = 8 with bias 127 the format's subnormal grid is a coarsening of
//     fp32's, so the bit-pattern rounding covers every magnitude (class INT);
//   * class GEN keeps values native (k = 0; every format value is an fp32
//     value) and rounds in fp64: the fp32 input fl32(x * 2^ft), or the sum of
//     two format values, is rounded on its fp64 bit pattern in the normal
//     range, onto the subnormal grid with the fp64 magic constant
//     2^(emin - m + 52) below it, and to INF from 2^(emax + 1) up.
// A sum of two format values whose magnitude is below 2^emin is a multiple
// of the smallest subnormal and so exact, and for m <= 10 an fp32 add
// followed by one rounding equals rounding the exact sum (24 >= 2(m+1) + 2,
// the double-rounding bound of Figueroa); wider mantissas add in fp64.
#pragma once

#include <stdint.h>

#include <cmath>

#include "aps.h"

namespace aps {

enum Cls : int32_t { CLS_INT = 0, CLS_TOP = 1, CLS_LOW = 2, CLS_GEN = 3 };
enum Acc : int32_t { ACC_F32 = 0, ACC_F64 = 1, ACC_EXACT = 2 };

// Kernel variants: one instantiation per (class, accumulator, m == 0).
enum Variant : int32_t {
    V_INT_F32 = 0,
    V_INT_F64 = 1,
    V_INT_EXACT = 2,
    V_INT_M0 = 3,
    V_TOP_F32 = 4,
    V_TOP_F64 = 5,
    V_TOP_M0 = 6,
    V_LOW_F32 = 7,
    V_LOW_F64 = 8,
    V_LOW_M0 = 9,
    V_GEN = 10,
    N_VARIANTS = 11
};

// Everything a kernel needs about one palette entry; built on the host.
struct FmtK {
    int32_t e, m, bias, emin, emax;
    int32_t k;        // working value = native value * 2^k
    int32_t j;        // LOW: subnormal rounding happens at working * 2^-j
    int32_t variant;  // Variant
    uint32_t sh;      // 23 - m: dropped fp32 mantissa bits
    uint32_t lsbw;    // width (0/1) of the tie bit read at position sh
    uint32_t half;    // increment added before the tie bit
    uint32_t mask;    // clears the dropped bits
    float thr;        // 2^emin in the working domain
    float c0;         // magic constant of the subnormal path (shifted by -j)
    float qs, qi;     // LOW: 2^Q and 2^-Q, Q = emin - m in the working domain (the subnormal step)
    uint32_t sh64;    // 52 - m  (fp64 accumulator)
    int32_t esh;      // max(0, -126 - emin): codes scale by 2^esh so that 2^emin is an fp32 normal
    uint64_t half64;  // 2^(sh64-1) - 1 (GEN with m = 0: 2^51, ties up)
    uint64_t mask64;  // clears the dropped fp64 bits
    double thr64;     // GEN: 2^emin
    double c064;      // GEN: 2^(emin - m + 52), the subnormal grid's magic constant
    double ovf64;     // GEN: 2^(emax + 1), where a rounded value is INF
    int32_t code_bits;
    int32_t emax_code;  // all-ones exponent field << m
};

// ------------------------------------------------------------------ host

inline int fmt_status(const aps_format& f) {
    if (f.e < 2 || f.e > 8 || f.m < 0 || f.m > 23) return APS_ERR_FORMAT;
    const int emin = 1 - f.bias;
    const int emax = (1 << f.e) - 2 - f.bias;
    if (emax > 127 || emin > emax || emin - f.m < -149) return APS_ERR_FORMAT;
    return APS_OK;
}

inline float pow2f_host(int p) {  // exact 2^p for -126 <= p <= 127
    union {
        uint32_t u;
        float f;
    } v;
    v.u = (uint32_t)(p + 127) << 23;
    return v.f;
}

inline FmtK make_fmtk(const aps_format& f) {
    FmtK o{};
    o.e = f.e;
    o.m = f.m;
    o.bias = f.bias;
    o.emin = 1 - f.bias;
    o.emax = (1 << f.e) - 2 - f.bias;
    const bool is_int = (f.e == 8 && f.bias == 127);
    // the shifted domain would leave part of the subnormal grid to fp32's underflow
    const bool is_gen = !is_int && (f.e == 8 || o.emin - f.m - 1 < -126);
    o.k = (is_int || is_gen) ? 0 : 127 - o.emax;
    const int emin_w = o.emin + o.k;
    o.sh = 23u - (uint32_t)f.m;
    if (f.m == 0) {  // ties of a 1-bit significand go to the even multiple: up
        o.half = 1u << 22;
        o.lsbw = 0;
    } else if (f.m == 23) {
        o.half = 0;
        o.lsbw = 0;
    } else {
        o.half = (1u << (o.sh - 1)) - 1u;
        o.lsbw = 1;
    }
    o.mask = ~((1u << o.sh) - 1u);
    o.thr = pow2f_host(emin_w < -126 ? -126 : emin_w);
    int cls;
    if (is_int) {
        cls = CLS_INT;
        o.j = 0;
        o.c0 = 0.f;
    } else if (is_gen) {
        cls = CLS_GEN;
        o.j = 0;
        o.c0 = 0.f;
    } else if (emin_w - f.m + 23 <= 127) {
        cls = CLS_TOP;
        o.j = 0;
        o.c0 = pow2f_host(emin_w - f.m + 23);
    } else {
        cls = CLS_LOW;
        o.j = emin_w - f.m + 23 - 127;
        o.c0 = pow2f_host(127);
        o.qs = pow2f_host(emin_w - f.m);
        o.qi = pow2f_host(f.m - emin_w);
    }
    int acc;
    if (is_int && f.m == 23)
        acc = ACC_EXACT;
    else if (f.m <= 10)
        acc = ACC_F32;
    else
        acc = ACC_F64;
    o.sh64 = 52u - (uint32_t)f.m;
    o.esh = o.emin < -126 ? -126 - o.emin : 0;
    o.half64 = (cls == CLS_GEN && f.m == 0) ? (1ull << 51) : (1ull << (o.sh64 - 1)) - 1ull;
    o.mask64 = ~((1ull << o.sh64) - 1ull);
    o.thr64 = std::ldexp(1.0, o.emin);
    o.c064 = std::ldexp(1.0, o.emin - f.m + 52);
    o.ovf64 = std::ldexp(1.0, o.emax + 1);
    if (cls == CLS_GEN)
        o.variant = V_GEN;
    else if (cls == CLS_INT)
        o.variant = f.m == 0 ? V_INT_M0 : (acc == ACC_EXACT ? V_INT_EXACT : (acc == ACC_F64 ? V_INT_F64 : V_INT_F32));
    else if (cls == CLS_TOP)
        o.variant = f.m == 0 ? V_TOP_M0 : (acc == ACC_F64 ? V_TOP_F64 : V_TOP_F32);
    else
        o.variant = f.m == 0 ? V_LOW_M0 : (acc == ACC_F64 ? V_LOW_F64 : V_LOW_F32);
    o.code_bits = 1 + f.e + f.m;
    o.emax_code = (int32_t)(((1u << f.e) - 1u) << f.m);
    return o;
}

// code container class: 0 nibble, 1 byte, 2 uint16, 3 none
inline int code_class(int bits) { return bits <= 4 ? 0 : (bits <= 8 ? 1 : (bits <= 16 ? 2 : 3)); }

}  // namespace aps
