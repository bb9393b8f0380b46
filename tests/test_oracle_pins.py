"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these compares the oracle with itself: each check uses the paper's
printed values (Table 2), an exact-rational enumeration of the format
(tests/exact_ref.py), a library routine that implements a special case
(numpy float16, torch bfloat16 / float8), or a closed-form property.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")

import oracle as O
from tests import exact_ref as X

F = O.Format
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

SMALL_FORMATS = [F(5, 2), F(4, 3), F(3, 0), F(2, 0), F(2, 1), F(3, 2), F(6, 1), F(3, 4),
                 F(4, 3, 5), F(5, 2, 20)]


def _fp32(v):
    return float(np.float32(v))


# ----------------------------------------------------- the formats modelled

FP32_MAX = (2 - Fraction(1, 2 ** 23)) * 2 ** 127
FP32_MIN_SUB = Fraction(1, 2 ** 149)


def test_format_ok_accepts_exactly_the_formats_fp32_holds():
    """A format is modelled when it has a sign, 2..8 exponent bits and 0..23
    mantissa bits and every one of its finite values is an fp32 value: its
    largest finite value (2 - 2^-m) * 2^emax at most fp32's, its smallest
    subnormal 2^(emin - m) at least fp32's 2^-149.  Values computed as exact
    rationals from the format's definition, across biases that put emax and
    emin - m on both sides of those limits."""
    for e in range(1, 10):
        for m in range(0, 25):
            dflt = (1 << (e - 1)) - 1
            top = (1 << e) - 2          # emax = top - bias
            biases = {dflt, dflt - 1, dflt + 1, top - 127, top - 128, top - 126, 150 - m, 149 - m, 151 - m, -5, 300}
            for bias in sorted(biases):
                emax, emin = top - bias, 1 - bias
                maxfinite = (2 - Fraction(1, 2 ** m)) * Fraction(2) ** emax
                minsub = Fraction(2) ** (emin - m)
                want = 2 <= e <= 8 and 0 <= m <= 23 and maxfinite <= FP32_MAX and minsub >= FP32_MIN_SUB
                assert O.format_ok(F(e, m, bias)) == want, (e, m, bias)


# ------------------------------------------------------------------ Table 2

def _table2():
    rows = []
    with open(os.path.join(GOLDEN, "table2_format_ranges.txt")) as fh:
        for line in fh:
            if line.strip() and not line.startswith("#"):
                name, e, m, lo, hi = line.split()
                rows.append((name, int(e), int(m), int(lo), int(hi)))
    return rows


@pytest.mark.parametrize("row", _table2(), ids=lambda r: r[0])
def test_table2_ranges(row):
    _, e, m, lo, hi = row
    f = F(e, m)
    assert O.format_ok(f)
    assert O.minsub(f) == 2.0 ** lo
    assert O.emax(f) == hi
    assert 2.0 ** hi <= O.maxfinite(f) < 2.0 ** (hi + 1)
    # the smallest value is kept, half of it is a tie that goes to zero,
    # anything above half of it rounds up to it
    assert O.round_(2.0 ** lo, f) == 2.0 ** lo
    assert O.round_(2.0 ** (lo - 1), f) == 0.0
    assert O.round_(2.0 ** (lo - 1) * (1 + 2.0 ** -20), f) == 2.0 ** lo
    # 2^hi is representable, 2^(hi+1) overflows to INF
    assert O.round_(2.0 ** hi, f) == 2.0 ** hi
    assert O.round_(2.0 ** (hi + 1), f) == math.inf
    assert O.round_(-(2.0 ** (hi + 1)), f) == -math.inf


def test_sec32_fp8_example():
    # 8 bits (exp 5, man 2): exponents in [-16, 15]; far above overflows, far below is 0
    f = F(5, 2)
    assert O.round_(2.0 ** 17, f) == math.inf
    assert O.round_(2.0 ** -18, f) == 0.0
    assert O.round_(2.0 ** 15, f) == 2.0 ** 15
    assert O.round_(2.0 ** -16, f) == 2.0 ** -16


# ------------------------------------------------- exhaustive enumeration

@pytest.mark.parametrize("f", SMALL_FORMATS, ids=str)
def test_codes_roundtrip_exhaustive(f):
    vals = X.values(f.e, f.m, f.b)
    nfin = len(vals)
    for code in range(1 << f.bits):
        sign = code >> (f.e + f.m)
        mag = code & ((1 << (f.e + f.m)) - 1)
        d = O.decode(code, f)
        if mag < nfin:
            ref = float(vals[mag]) * (-1.0 if sign else 1.0)
            assert d == ref and math.copysign(1.0, d) == (-1.0 if sign else 1.0), code
            assert O.round_(d, f) == d
            assert O.encode(d, f) == code
        elif mag == nfin:  # exponent all ones, mantissa zero
            assert d == (-math.inf if sign else math.inf)
            assert O.encode(d, f) == code
        else:
            assert math.isnan(d)


@pytest.mark.parametrize("f", SMALL_FORMATS, ids=str)
def test_round_midpoints_exhaustive(f):
    """Every midpoint between neighbours (and beyond the largest value), and
    the fp32 values one ulp either side of it, round as the exact reference."""
    vals = list(X.values(f.e, f.m, f.b)) + [Fraction(2) ** (O.emax(f) + 1)]
    for lo, hi in zip(vals[:-1], vals[1:]):
        mid = float((lo + hi) / 2)
        for y in (mid, np.nextafter(np.float32(mid), np.float32(0)),
                  np.nextafter(np.float32(mid), np.float32(np.inf))):
            y = float(y)
            for s in (1.0, -1.0):
                got = O.round_(s * y, f)
                ref = X.round_exact(s * y, f.e, f.m, f.b)
                assert got == float(ref), (f, s * y, got, ref)


@pytest.mark.parametrize("f", SMALL_FORMATS + [F(5, 10), F(8, 7), F(6, 9), F(7, 5)], ids=str)
def test_round_random_fp32(f):
    rng = np.random.default_rng(1911)
    # magnitudes log-uniform across and beyond the format's range, plus fp32 subnormals
    lo, hi = math.log2(O.minsub(f)) - 4, O.emax(f) + 3
    ex = rng.uniform(lo, hi, 1500)
    ys = (rng.choice([-1, 1], 1500) * 2.0 ** ex).astype(np.float32)
    ys = np.concatenate([ys, np.array([1e-45, -3e-44, 1e-39, 0.0, -0.0], np.float32)])
    for y in ys:
        got = O.round_(float(y), f)
        ref = X.round_exact(float(y), f.e, f.m, f.b)
        assert got == float(ref), (f, float(y), got, ref)
        if got == 0.0:  # an underflow keeps the sign of the input
            assert math.copysign(1, got) == math.copysign(1, float(y))


@pytest.mark.parametrize("f", [F(5, 2), F(4, 3), F(3, 0), F(2, 1), F(3, 2)], ids=str)
def test_pairwise_rounded_add_exhaustive(f):
    """R(a + b) for every pair of finite codes equals rounding the exact sum."""
    vals = X.values(f.e, f.m, f.b)
    fv = [float(v) for v in vals]
    fv = fv + [-v for v in fv[1:]]
    fr = [Fraction(v) for v in fv]
    for a, fa in zip(fv, fr):
        for b, fb in zip(fv, fr):
            got = O.round_(a + b, f)
            t = fa + fb
            ref = X.round_exact(t, f.e, f.m, f.b) if t != 0 else Fraction(0)
            assert got == float(ref), (f, a, b)


# ------------------------------------------------- library special cases

def test_fp16_equals_numpy_half():
    rng = np.random.default_rng(7)
    y = (rng.choice([-1, 1], 200000) * 2.0 ** rng.uniform(-30, 17, 200000)).astype(np.float32)
    ref = y.astype(np.float16).astype(np.float64)
    got = O.round_array(y, F(5, 10))
    assert np.array_equal(got, ref)


def test_bf16_equals_torch_bfloat16():
    rng = np.random.default_rng(8)
    y = (rng.choice([-1, 1], 100000) * 2.0 ** rng.uniform(-140, 127.99, 100000)).astype(np.float32)
    ref = torch.from_numpy(y).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.round_array(y, F(8, 7))
    assert np.array_equal(got, ref)


def test_e5m2_equals_torch_float8_e5m2():
    rng = np.random.default_rng(9)
    y = (rng.choice([-1, 1], 100000) * 2.0 ** rng.uniform(-19, 17, 100000)).astype(np.float32)
    ref = torch.from_numpy(y).to(torch.float8_e5m2).to(torch.float64).numpy()
    got = O.round_array(y, F(5, 2))
    assert np.array_equal(got, ref)


def test_e4m3_equals_torch_float8_e4m3fn_below_248():
    # e4m3fn spends the all-ones exponent on finite values; below 248 the two agree
    rng = np.random.default_rng(10)
    y = (rng.choice([-1, 1], 100000) * 2.0 ** rng.uniform(-12, 7.95, 100000)).astype(np.float32)
    y = y[np.abs(y) < 248]
    ref = torch.from_numpy(y).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = O.round_array(y, F(4, 3))
    assert np.array_equal(got, ref)


def test_fp32_format_is_identity():
    rng = np.random.default_rng(11)
    y = rng.standard_normal(20000).astype(np.float32) * np.float32(1e-30)
    y = np.concatenate([y, np.array([3.4e38, 1e-45, 1.17e-38], np.float32)])
    got = O.round_array(y, F(8, 23))
    assert np.array_equal(got, y.astype(np.float64))


def test_sum_fp16_equals_numpy_sequential():
    rng = np.random.default_rng(12)
    W, n = 16, 3000
    G = (rng.standard_normal((W, n)) * 2.0 ** rng.uniform(-20, 10, (W, 1))).astype(np.float32)
    offs = np.array([0, n], np.int64)
    got = O.sim_reduce(G, n, offs, None, F(5, 10))
    s = G[0].astype(np.float16)
    for w in range(1, W):
        s = (s + G[w].astype(np.float16)).astype(np.float16)
    assert np.array_equal(got, s.astype(np.float32))


def test_sum_fp32_equals_sequential_float32():
    rng = np.random.default_rng(13)
    W, n = 9, 4000
    G = (rng.standard_normal((W, n)) * 2.0 ** rng.uniform(-50, 50, (W, n))).astype(np.float32)
    offs = np.array([0, n], np.int64)
    got = O.sim_reduce(G, n, offs, None, F(8, 23))
    s = G[0].copy()
    for w in range(1, W):
        s = (s + G[w]).astype(np.float32)
    assert np.array_equal(got, s)


# ---------------------------------------------------------------- scales

def test_scale_worked_example():
    # 1-5-2, N = 8, max |g| = 0.1: fl32(0.8) in (0.5, 1] so ceil(log2) = 0 and
    # the scale exponent is emax - 0 = 15 (closed form of Sec. 3.3.3)
    bits = int(np.float32(0.1).view(np.uint32))
    assert O.scale_one(bits, 8, F(5, 2)) == 15
    # a power of two: N * ghat = 2^-3 exactly -> ceil(log2) = -3 -> 15 + 3
    bits = int(np.float32(2.0 ** -6).view(np.uint32))
    assert O.scale_one(bits, 8, F(5, 2)) == 18


def test_scale_special_cases():
    f = F(5, 2)
    assert O.scale_one(0, 8, f) == 0
    assert O.scale_one(0x7F800000, 8, f) == 0
    assert O.scale_one(0x7FC00000, 8, f) == 0
    assert O.scale_one(int(np.float32(3e38).view(np.uint32)), 8, f) == 0  # N*g overflows
    assert O.scale_one(1, 1, f) == 15 + 149  # smallest fp32 subnormal


def test_scale_maximality_and_closed_form():
    """N*ghat*2^f lies in (2^(emax-1), 2^emax]: the largest power of two that
    keeps the relaxed bound of Eq. (2)-(3); checked against exact rationals."""
    rng = np.random.default_rng(14)
    for f in (F(5, 2), F(4, 3), F(8, 7), F(3, 0), F(5, 10), F(4, 3, 5)):
        em = O.emax(f)
        for _ in range(400):
            g = np.float32(2.0 ** rng.uniform(-149, 100) * rng.uniform(1, 2))
            N = int(rng.choice([1, 2, 3, 7, 8, 100, 256, 1000, 65536]))
            t = np.float32(np.float32(N) * g)
            if not np.isfinite(t) or t == 0:
                continue
            ft = O.scale_one(int(g.view(np.uint32)), N, f)
            assert ft == em - X.ceil_log2_exact(Fraction(float(t)))
            v = Fraction(float(t)) * Fraction(2) ** ft
            assert Fraction(2) ** (em - 1) < v <= Fraction(2) ** em


def test_scale_matches_literal_findmaxexp():
    """Algorithm 1 literally (FindMaxExp(g*N) per worker, then MAX over workers,
    then upper_bound_exp - max) equals scales computed from the max magnitude."""
    rng = np.random.default_rng(15)
    for f in (F(5, 2), F(4, 3), F(3, 0), F(8, 7)):
        ub = 2 ** (f.e - 1) - 1
        for N in (2, 3, 8, 12):
            W, n = N, 500
            G = (rng.standard_normal((W, n)) * 2.0 ** rng.uniform(-40, 20)).astype(np.float32)
            G[:, rng.random(n) < 0.1] = 0
            G[:, 400:450] = 0                      # an all-zero layer: no exponent, scale 0
            offs = np.array([0, 123, 123, 400, 450, n], np.int64)
            mb = O.layer_maxabs(G, n, offs)
            se = O.layer_scales(mb, N, f)
            for i in range(len(offs) - 1):
                exps = [O.find_max_exp(G[w, offs[i]:offs[i + 1]], N)[0] for w in range(W)]
                mx = max(exps)
                lit = 0 if mx == -2 ** 31 else ub - mx
                assert se[i] == lit, (f, N, i)
    # a zero has no exponent; INF and NaN products are reported apart
    assert O.find_max_exp(np.zeros(3, np.float32), 8) == (-2 ** 31, False)
    assert O.find_max_exp(np.array([0.0, 3.0, np.inf], np.float32), 2) == (3, True)
    assert O.find_max_exp(np.array([np.nan, -0.75], np.float32), 1) == (0, True)


def test_maxabs_nan_inf_zero():
    G = np.zeros((3, 12), np.float32)
    offs = np.array([0, 4, 8, 12], np.int64)
    G[1, 1] = -2.5
    G[2, 5] = np.inf
    G[0, 6] = 1e30
    G[1, 9] = np.nan
    G[2, 10] = -1e38
    mb = O.layer_maxabs(G, 12, offs)
    assert mb[0] == np.float32(2.5).view(np.uint32)
    assert mb[1] == 0x7F800000
    assert mb[2] > 0x7F800000


# ------------------------------------------------- brute force W-way sums

@pytest.mark.parametrize("f", [F(3, 0), F(4, 3), F(5, 2), F(2, 1), F(4, 3, 5)], ids=str)
@pytest.mark.parametrize("mode", ["aps", "raw"])
def test_sim_reduce_brute_force(f, mode):
    rng = np.random.default_rng(16 + f.e * 7 + f.m)
    for trial in range(6):
        W = int(rng.integers(1, 9))
        n = int(rng.integers(1, 65))
        scales = 2.0 ** rng.uniform(-8, 3, W)[:, None]
        G = (rng.standard_normal((W, n)) * scales).astype(np.float32)
        G[rng.random((W, n)) < 0.1] = 0
        cut = int(rng.integers(0, n + 1))
        offs = np.array([0, cut, n], np.int64)
        if mode == "aps":
            mb = O.layer_maxabs(G, n, offs)
            # scale from exact rationals, independent of the oracle's own routine
            se = []
            for i in range(2):
                gh = np.uint32(mb[i]).view(np.float32)
                t = np.float32(np.float32(W) * gh)
                se.append(0 if gh == 0 else O.emax(f) - X.ceil_log2_exact(Fraction(float(t))))
            se = np.array(se, np.int32)
        else:
            se = None
        got = O.sim_reduce(G, n, offs, se, f)
        for i in range(2):
            ft = 0 if se is None else int(se[i])
            for j in range(offs[i], offs[i + 1]):
                qs = [X.round_exact(Fraction(float(np.float32(math.ldexp(float(G[w, j]), ft)))),
                                    f.e, f.m, f.b) for w in range(W)]
                s = X.sum_exact(qs, f.e, f.m, f.b)
                ref = float(s) * 2.0 ** -ft if not isinstance(s, float) else s
                assert got[j] == np.float32(ref) or (math.isnan(ref) and math.isnan(got[j])), \
                    (f, mode, trial, j, got[j], ref)


def test_zero_sign_rules():
    f = F(5, 2)
    offs = np.array([0, 4], np.int64)
    G = np.array([[1.0, -0.0, -1e-9, 2.0], [-1.0, -0.0, -1e-9, -0.0]], np.float32)
    got = O.sim_reduce(G, 4, offs, None, f)
    assert [math.copysign(1, v) for v in got] == [1, -1, -1, 1]
    assert got[0] == 0 and got[1] == 0 and got[2] == 0 and got[3] == 2.0


# ------------------------------------------------------------ invariants

def _synthetic(rng, W, n, lo=-7, hi=-1):
    G = (rng.standard_normal((W, n)) * 10.0 ** rng.uniform(lo, hi)).astype(np.float32)
    G[rng.random((W, n)) < 0.02] = 0
    out = rng.random((W, n)) < 1e-3
    G[out] *= 100
    return G


def test_aps_mode_never_overflows():
    rng = np.random.default_rng(17)
    for f in (F(5, 2), F(4, 3), F(3, 0), F(2, 1)):
        for W in (1, 2, 3, 8, 13, 64):
            n = 700
            G = _synthetic(rng, W, n)
            offs = np.array([0, 10, 300, n], np.int64)
            se = O.layer_scales(O.layer_maxabs(G, n, offs), W, f)
            out = O.sim_reduce(G, n, offs, se, f)
            assert np.all(np.isfinite(out)), (f, W)
            scaled = O.sim_reduce(G, n, offs, se, f, flags=O.OUTPUT_SCALED)
            assert np.all(np.abs(scaled) <= 2.0 ** O.emax(f))


def test_power_of_two_scaling_is_exact():
    """Scaling by 2^k moves only the exponent (Sec. 3.3.1): within the
    format's normal range, quantising at scale k and unscaling equals
    rounding the significand directly (numpy float16 as the m = 10 route)."""
    rng = np.random.default_rng(18)
    x = (rng.standard_normal(5000) * 3e-6).astype(np.float32)
    x = x[np.abs(x) > 2e-8]
    n = x.size
    offs = np.array([0, n], np.int64)
    k = 20  # |x| * 2^20 stays inside the fp16 normal range
    Q = O.quantize(x[None, :], n, offs, np.array([k], np.int32), F(5, 10))
    back = O.dequantize(Q[0], None, n, offs, np.array([k], np.int32), F(5, 10))
    direct = (x * np.float32(2.0 ** k)).astype(np.float16).astype(np.float32) / np.float32(2.0 ** k)
    assert np.array_equal(back, direct)
    # and a power-of-two round trip leaves an fp32 value unchanged
    assert np.array_equal(np.ldexp(np.ldexp(x, 37), -37), x)


@pytest.mark.parametrize("f", [F(5, 2), F(4, 3), F(3, 0), F(5, 10)], ids=str)
def test_round_properties(f):
    rng = np.random.default_rng(19)
    ys = np.sort(np.abs((rng.standard_normal(3000) * 2.0 ** rng.uniform(-20, 18, 3000))))
    r = O.round_array(ys, f)
    assert np.all(r[1:] >= r[:-1])                                        # monotone
    assert np.array_equal(O.round_array(r, f), r)                         # idempotent
    assert np.array_equal(O.round_array(-ys, f), -r)                      # odd
    fin = np.isfinite(r)
    assert all(O.encode(v, f) < (1 << f.bits) for v in r[fin][:200])      # encodable


def test_w1_reduce_is_quantize_dequantize_and_composition():
    rng = np.random.default_rng(20)
    n = 900
    offs = np.array([0, 5, 5, 400, n], np.int64)
    for f in (F(5, 2), F(4, 3), F(3, 0)):
        G = _synthetic(rng, 6, n)
        se = O.layer_scales(O.layer_maxabs(G, n, offs), 6, f)
        # W = 1
        r1 = O.sim_reduce(G[:1], n, offs, se, f)
        q1 = O.quantize(G[:1], n, offs, se, f)
        d1 = O.dequantize(q1[0], None, n, offs, se, f)
        assert np.array_equal(r1, d1)
        # fused == composition dequantize(sim_reduce(quantize(x), IN_Q|OUT_SCALED))
        full = O.sim_reduce(G, n, offs, se, f)
        Q = O.quantize(G, n, offs, se, f)
        red = O.sim_reduce(Q, n, offs, se, f, flags=O.INPUT_QUANTIZED | O.OUTPUT_SCALED)
        comp = O.dequantize(red, None, n, offs, se, f)
        assert np.array_equal(full, comp)
        # codes carry the same values
        codes = O.pack_codes(red, offs, f)
        comp2 = O.dequantize(None, codes, n, offs, se, f)
        assert np.array_equal(full, comp2)


def test_code_layout_against_library_bit_patterns():
    """The packed code layout of the header (code = sign, exponent field,
    mantissa; 9..16-bit codes as little-endian uint16, 5..8-bit codes one
    byte each, 2..4-bit codes two per byte with element 2i in the low
    nibble), pinned to bit patterns the oracle does not produce: numpy's
    IEEE half for 1-5-10, torch's float8_e5m2 for 1-5-2, and, for 4-bit
    codes, values built from each code by the format's definition."""
    rng = np.random.default_rng(515)
    # 1-5-10 is IEEE half precision: its codes are float16 bit patterns
    h = (rng.standard_normal(2000) * 2.0 ** rng.integers(-26, 16, 2000)).astype(np.float16)
    h[:6] = [0.0, -0.0, np.inf, -np.inf, 6.1035e-05, -5.96e-08]  # 2^-14, -2^-24
    v = h.astype(np.float32)
    assert np.array_equal(v.astype(np.float16).view(np.uint16), h.view(np.uint16))
    offs = np.array([0, v.size], np.int64)
    assert O.pack_codes(v, offs, F(5, 10)).tobytes() == h.astype("<f2").tobytes()
    # 1-5-2 is float8_e5m2: one byte per code (NaN is not compared: torch writes another pattern)
    x = torch.from_numpy(rng.standard_normal(2000).astype(np.float32) * 2.0 ** 8)
    x[:4] = torch.tensor([0.0, -0.0, float("inf"), -float("inf")])
    e5 = x.to(torch.float8_e5m2)
    v8 = e5.to(torch.float32).numpy()
    offs = np.array([0, v8.size], np.int64)
    assert np.array_equal(O.pack_codes(v8, offs, F(5, 2)), e5.view(torch.uint8).numpy())
    # 4-bit codes of 1-3-0 (bias 3) and 1-2-1 (bias 1): every code's value from the definition
    for f, bias in ((F(3, 0), 3), (F(2, 1), 1)):
        emask = (1 << f.e) - 1
        codes = rng.integers(0, 16, 601)
        vals = []
        for c in codes:
            sign = -1.0 if c >> (f.e + f.m) else 1.0
            ef, mant = (c >> f.m) & emask, c & ((1 << f.m) - 1)
            if ef == emask:
                codes[len(vals)] = c = c & ~((1 << f.m) - 1)  # INF only: NaN's mantissa is checked below
                vals.append(sign * np.inf)
            elif ef == 0:
                vals.append(sign * mant * 2.0 ** (1 - bias - f.m))
            else:
                vals.append(sign * (1 + mant / 2 ** f.m) * 2.0 ** (ef - bias))
        vals = np.array(vals, np.float32)
        offs = np.array([0, vals.size], np.int64)
        packed = O.pack_codes(vals, offs, f)
        c = np.append(codes, 0).astype(np.uint8)
        assert np.array_equal(packed, c[0::2] | (c[1::2] << 4)), f
    # NaN: the all-ones exponent with the top mantissa bit (the INF code when m = 0)
    assert O.encode(float("nan"), F(5, 10)) & 0x7FFF == 0x7E00
    assert O.encode(float("nan"), F(5, 2)) & 0x7F == 0x7E
    assert O.encode(float("nan"), F(4, 3)) & 0x7F == 0x7C
    assert O.encode(float("nan"), F(3, 0)) & 0x7 == 0x7


def test_raw_mode_overflow_and_nan():
    f = F(5, 2)
    offs = np.array([0, 4], np.int64)
    G = np.array([[7e4, -7e4, np.nan, 5e4], [7e4, 7e4, 1.0, 5e4]], np.float32)
    out = O.sim_reduce(G, 4, offs, None, f)
    assert out[0] == np.inf          # INF + INF
    assert np.isnan(out[1])          # -INF + INF
    assert np.isnan(out[2])          # NaN propagates
    assert out[3] == np.inf          # 49152 + 49152 = 98304 > 61440 -> INF


# --------------------------------------------------- reduce of packed codes

def _pack(codes_rows, bits):
    """Pack W rows of integer codes (independent of the oracle's packer)."""
    W, n = codes_rows.shape
    if bits <= 4:
        rb = (n + 1) // 2
        out = np.zeros((W, rb), np.uint8)
        for w in range(W):
            for j in range(n):
                out[w, j // 2] |= (int(codes_rows[w, j]) & 15) << (4 * (j % 2))
    elif bits <= 8:
        out = codes_rows.astype(np.uint8)
    else:
        out = codes_rows.astype("<u2").view(np.uint8).reshape(W, -1)
    return out


@pytest.mark.parametrize("f", [F(3, 0), F(4, 3), F(5, 2), F(2, 1), F(5, 10)], ids=str)
def test_sim_reduce_codes_brute_force(f):
    rng = np.random.default_rng(30 + f.e + f.m)
    vals = X.values(f.e, f.m, f.b)
    nfin = len(vals)
    for trial in range(5):
        W = int(rng.integers(1, 9))
        n = int(rng.integers(2, 41)) // 2 * 2
        # finite codes only (INF/NaN arithmetic is covered elsewhere)
        mags = rng.integers(0, nfin, (W, n))
        signs = rng.integers(0, 2, (W, n))
        codes = mags | (signs << (f.e + f.m))
        packed = _pack(codes, f.bits)
        offs = np.array([0, n // 2, n], np.int64)
        got = O.sim_reduce_codes(packed, W, n, n, offs, None, f, flags=O.OUTPUT_SCALED)
        for j in range(n):
            qs = [(-1 if signs[w, j] else 1) * vals[mags[w, j]] for w in range(W)]
            ref = X.sum_exact(qs, f.e, f.m, f.b)
            assert got[j] == float(ref), (f, trial, j)


# ----------------------------------------- summation orders and Kahan (Sec. 4.2, 5)

@pytest.mark.parametrize("f", [F(5, 2), F(4, 3), F(3, 0)], ids=str)
@pytest.mark.parametrize("acc", [O.ACC_SEQUENTIAL, O.ACC_KAHAN])
def test_ordered_reduce_brute_force(f, acc):
    rng = np.random.default_rng(50 + f.e + 7 * acc)
    for W, k in ((4, 1), (4, 2), (8, 2), (8, 4), (8, 8), (6, 3), (3, 1)):
        n = 24
        G = (rng.standard_normal((W, n)) * 2.0 ** rng.uniform(-4, 2, (W, 1))).astype(np.float32)
        offs = np.array([0, n], np.int64)
        got = O.sim_reduce_ex(G, n, offs, None, f, group=k, accumulator=acc)
        ng = W // k
        for j in range(n):
            qs = [X.round_exact(Fraction(float(G[w, j])), f.e, f.m, f.b) for w in range(W)]
            if any(isinstance(q, float) for q in qs):
                continue
            ref = X.hierarchical_exact(qs, k, j * ng // n, f.e, f.m, f.b, kahan=(acc == O.ACC_KAHAN))
            if isinstance(ref, float):
                assert got[j] == ref, (f, W, k, j)
            else:
                assert got[j] == float(ref), (f, W, k, acc, j, got[j], float(ref))


def test_kahan_recovers_what_plain_loses():
    # 1-5-10: 1 + 2^-11 is a tie that rounds back to 1, so a plain low-precision
    # accumulator never moves; the exact sum of 1 and 2048 * 2^-11 is 2
    W, n = 2049, 1
    G = np.full((W, 4), 2.0 ** -11, np.float32)
    G[0, :] = 1.0
    offs = np.array([0, n], np.int64)
    plain = O.sim_reduce_ex(G, n, offs, None, F(5, 10), accumulator=O.ACC_SEQUENTIAL)
    kahan = O.sim_reduce_ex(G, n, offs, None, F(5, 10), accumulator=O.ACC_KAHAN)
    assert plain[0] == 1.0
    assert kahan[0] == 2.0


def test_kahan_error_bound_fp32():
    # Kahan's bound for the fp32 format: |sum - exact| <= (2u + O(W u^2)) * sum |x|
    rng = np.random.default_rng(51)
    W, n = 1000, 64
    G = (rng.standard_normal((W, n)) * 10.0 ** rng.uniform(-3, 3, (W, n))).astype(np.float32)
    offs = np.array([0, n], np.int64)
    got = O.sim_reduce_ex(G, n, offs, None, F(8, 23), accumulator=O.ACC_KAHAN)
    u = 2.0 ** -24
    for j in range(n):
        exact = sum(Fraction(float(v)) for v in G[:, j])
        absum = sum(abs(Fraction(float(v))) for v in G[:, j])
        err = abs(Fraction(float(got[j])) - exact)
        assert err <= (2 * u + 4 * W * u * u) * absum + Fraction(abs(float(exact))) * u


def test_order_special_cases():
    rng = np.random.default_rng(52)
    W, n = 8, 50
    G = rng.standard_normal((W, n)).astype(np.float32)
    offs = np.array([0, 20, n], np.int64)
    f = F(5, 2)
    se = np.array([3, -2], np.int32)
    # one group of W workers is the plain worker order
    assert np.array_equal(O.sim_reduce_ex(G, n, offs, se, f, group=W), O.sim_reduce(G, n, offs, se, f))
    # any order of the fp32 format with exact adds: integers sum exactly
    Gi = rng.integers(-1000, 1000, (W, n)).astype(np.float32)
    ring = O.sim_reduce_ex(Gi, n, offs, None, F(8, 23), group=1)
    assert np.array_equal(ring, Gi.sum(0))


def test_round_off_error_eq5():
    h = np.array([1.0, 2.0, 0.0, 4.0], np.float32)
    l = np.array([1.5, 2.0, 7.0, 3.0], np.float32)
    # (0.5 + 0 + 0.25) / 3, the zero entry of grad_h left out
    assert O.round_off_error(h, l) == pytest.approx(0.25, abs=0)


# ------------------------------- low-precision-accumulator GEMM (Sec. 5, CPD)

def _gemm_exact(A, B, fin, facc, kahan):
    """Exact-rational reference: inputs cast to fin, each product cast to facc,
    the products of an output chained in k order in facc.  INF and NaN pass
    through Python float arithmetic (IEEE)."""
    M, K = A.shape
    N = B.shape[1]
    out = np.zeros((M, N))
    for i in range(M):
        for j in range(N):
            ps = []
            for k in range(K):
                a = X.round_exact(Fraction(float(A[i, k])), fin.e, fin.m, fin.b)
                b = X.round_exact(Fraction(float(B[k, j])), fin.e, fin.m, fin.b)
                ps.append(X.round_exact(a * b, facc.e, facc.m, facc.b))
            out[i, j] = float(X.chain_exact(ps, facc.e, facc.m, facc.b, kahan=kahan))
    return out


@pytest.mark.parametrize("fin,facc", [(F(5, 2), F(5, 2)), (F(4, 3), F(5, 2)), (F(5, 2), F(4, 3)),
                                      (F(2, 1), F(3, 0)), (F(2, 0), F(2, 0)), (F(3, 2), F(4, 3, 5))],
                         ids=lambda f: str(f))
@pytest.mark.parametrize("acc", [O.ACC_SEQUENTIAL, O.ACC_KAHAN])
def test_lp_gemm_brute_force(fin, facc, acc):
    rng = np.random.default_rng(60 + fin.e + 3 * facc.m + 11 * acc)
    # magnitudes over the input format's range, from below its smallest
    # subnormal to about the square root of its largest value
    lo, hi = O.emin(fin) - fin.m - 1, max(O.emax(fin) // 2, 1)
    finite = 0
    for M, N, K in ((3, 4, 7), (2, 2, 1), (1, 3, 12), (4, 2, 5)):
        A = (rng.standard_normal((M, K)) * 2.0 ** rng.uniform(lo, hi, (M, K))).astype(np.float32)
        B = (rng.standard_normal((K, N)) * 2.0 ** rng.uniform(lo, hi, (K, N))).astype(np.float32)
        got = O.lp_gemm(A, B, fin, facc, acc)
        ref = _gemm_exact(A, B, fin, facc, acc == O.ACC_KAHAN)
        same = (got == ref) | (np.isnan(got) & np.isnan(ref))
        assert same.all(), (fin, facc, acc, M, N, K, got, ref)
        finite += int(np.isfinite(ref).sum())
    assert finite >= 10


def test_lp_gemm_fp32_accumulator_is_a_float32_dot_product():
    # products of fp16 values are exact in fp32, so with the fp32 format as the
    # accumulator each output is numpy's float32 dot product taken in k order
    rng = np.random.default_rng(61)
    M, N, K = 5, 6, 40
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = (rng.standard_normal((K, N)) * 100).astype(np.float32)
    got = O.lp_gemm(A, B, F(5, 10), F(8, 23))
    a = A.astype(np.float16).astype(np.float32)
    b = B.astype(np.float16).astype(np.float32)
    for i in range(M):
        for j in range(N):
            s = np.float32(a[i, 0] * b[0, j])
            for k in range(1, K):
                s = np.float32(s + np.float32(a[i, k] * b[k, j]))
            assert got[i, j] == s


def test_lp_gemm_fp16_equals_numpy_float16_arithmetic():
    # numpy float16 multiplies and adds round their exact result to float16
    # (through float32, which is innocuous: 24 >= 2 * 11 + 2)
    rng = np.random.default_rng(62)
    M, N, K = 4, 5, 64
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = (rng.standard_normal((K, N)) * 8).astype(np.float32)
    got = O.lp_gemm(A, B, F(5, 10), F(5, 10))
    a = A.astype(np.float16)
    b = B.astype(np.float16)
    for i in range(M):
        for j in range(N):
            s = a[i, 0] * b[0, j]
            for k in range(1, K):
                s = np.float16(s + a[i, k] * b[k, j])
            assert got[i, j] == np.float32(s)


def test_lp_gemm_bf16_equals_torch_bfloat16_arithmetic():
    rng = np.random.default_rng(63)
    M, N, K = 6, 7, 50
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = (rng.standard_normal((K, N)) * 3).astype(np.float32)
    got = O.lp_gemm(A, B, F(8, 7), F(8, 7))
    a = torch.from_numpy(A).to(torch.bfloat16)
    b = torch.from_numpy(B).to(torch.bfloat16)
    s = a[:, 0:1] * b[0:1, :]
    for k in range(1, K):
        s = s + a[:, k:k + 1] * b[k:k + 1, :]
    assert np.array_equal(got, s.to(torch.float32).numpy())


@pytest.mark.parametrize("f", [F(5, 2), F(4, 3), F(5, 10), F(3, 1)], ids=str)
def test_lp_gemm_swamping_closed_form(f):
    # a sum of ones in a p-bit significand grows to 2^p and stops there: 2^p + 1
    # is a tie between 2^p (even) and 2^p + 2 -- the loss Sec. 5 describes
    p = f.m + 1
    for K in (1, 2, 2 ** p - 1, 2 ** p, 2 ** p + 1, 2 ** p + 7, 3 * 2 ** p):
        if K > O.maxfinite(f):
            continue
        got = O.lp_gemm(np.ones((1, K), np.float32), np.ones((K, 1), np.float32), f, f)
        assert got[0, 0] == min(K, 2 ** p), (f, K)
        # Kahan keeps the running sum within one quantum of K
        kah = O.lp_gemm(np.ones((1, K), np.float32), np.ones((K, 1), np.float32), f, f, O.ACC_KAHAN)
        quantum = 2.0 ** (max(math.floor(math.log2(K)), 0) - f.m)
        assert abs(kah[0, 0] - K) <= quantum, (f, K, kah[0, 0])


def test_lp_gemm_transpose_and_edge_shapes():
    rng = np.random.default_rng(64)
    A = rng.standard_normal((5, 9)).astype(np.float32)
    B = rng.standard_normal((9, 3)).astype(np.float32)
    for acc in (O.ACC_SEQUENTIAL, O.ACC_KAHAN):
        C = O.lp_gemm(A, B, F(4, 3), F(5, 2), acc)
        Ct = O.lp_gemm(np.ascontiguousarray(B.T), np.ascontiguousarray(A.T), F(4, 3), F(5, 2), acc)
        assert np.array_equal(C, Ct.T)
    # K = 0: the empty sum is +0
    Z = O.lp_gemm(np.zeros((2, 0), np.float32), np.zeros((0, 3), np.float32), F(5, 2), F(5, 2))
    assert np.array_equal(Z, np.zeros((2, 3))) and not np.signbit(Z).any()
