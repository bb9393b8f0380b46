"""The claim behind aps_sync's one-pass route, checked on the CPU with a
small numpy model of that route against the oracle.

Power-of-two scaling commutes with rounding to m+1 significant bits
(Sec. 3.3.1).  So the W-worker sum rounded after every add (Algorithm 1 with
the low-precision accumulator of Sec. 5) can be formed on the UNSCALED
values, with the rounding's exponent unbounded, before the layer's scale
2^ft is known.  With T = max(2^(emin - ft), 2^-126), N = W a power of two,
m <= 10 and a layer with 0 < N * ghat <= 2^127 (or ghat = 0), the unscaled
chain equals the oracle's result, unscaled, for every element in which each
nonzero input x_k either has |x_k| >= T, or arrives (k >= 1) when the
unscaled partial sum has |s_(k-1)| >= 2^(m+3) * T, so that both chains
leave the sum unchanged.  The route keeps, per element, the exponent of
min_k max(|x_k|, |s_(k-1)| * 2^-(m+3)) (zeros skipped) and recomputes the
element when it lies below T.  The model below implements that route (fp32
adds, rounding on fp32 bit patterns, the per-element byte and the per-layer
threshold) in numpy; it shares nothing with the HIP library or the oracle.
The tests check that every element the criterion accepts matches the oracle
bit for bit, and that elements it rejects do differ in some of the cases
(so the recomputation is needed and the test can fail).  They also check
what lets the route keep its sums in 2 bytes for m <= 7: an accepted sum is
a multiple of 2^(-126 - m), so the low 16 bits of its fp32 pattern are
zero."""
import numpy as np
import pytest

import oracle as O
from tests._util import ofmt
from tests.sync_cases import LAYER_MAXIMA, threshold_values
from paper_1911_08907_amd.aps import Format as F


def _rho(b: np.ndarray, m: int) -> np.ndarray:
    """Round fp32 bit patterns to m+1 significant bits, exponent unbounded:
    ties to the even significand; m = 0 ties up (the even multiple)."""
    sh = np.uint32(23 - m)
    if m == 0:
        half, lw = np.uint32(1 << 22), np.uint32(0)
    else:
        half, lw = np.uint32((1 << (22 - m)) - 1), np.uint32(1)
    mask = np.uint32(~((1 << (23 - m)) - 1) & 0xFFFFFFFF)
    with np.errstate(over="ignore"):
        return ((b + half + ((b >> sh) & lw)) & mask).astype(np.uint32)


def model(G, n, offs, f, W, scale_exp, maxabs):
    """The one-pass route: unscaled rounded sums, exponent bytes, per-layer
    thresholds; returns (sums, flagged)."""
    X = np.ascontiguousarray(G[:, :n]).view(np.uint32)
    ab = X & np.uint32(0x7FFFFFFF)
    one = np.uint32(1)
    sc = np.float32(2.0 ** -(f.m + 3))
    s = _rho(X[0], f.m).view(np.float32)
    with np.errstate(over="ignore"):
        mn = ab[0] - one                          # a zero wraps to the top
    for w in range(1, W):
        # the term's magnitude, or the sum it meets scaled down by 2^(m+3)
        c = (np.abs(s) * sc).astype(np.float32).view(np.uint32)
        with np.errstate(over="ignore"):
            mn = np.minimum(mn, np.maximum(ab[w] - one, c))
        q = _rho(X[w], f.m).view(np.float32)
        with np.errstate(over="ignore", invalid="ignore"):
            t = (s + q).astype(np.float32)
        s = _rho(t.view(np.uint32), f.m).view(np.float32)
    byte = np.minimum(mn >> np.uint32(23), np.uint32(255)).astype(np.int32)
    emin, emax = 1 - f.b, (1 << f.e) - 2 - f.b
    L = offs.size - 1
    thr = np.full(L, 256, np.int32)
    for i in range(L):
        g = int(maxabs[i]) & 0x7FFFFFFF
        if g == 0:
            thr[i] = 0
        elif g < 0x7F800000:
            with np.errstate(over="ignore"):
                t = np.float32(W) * np.array([g], np.uint32).view(np.float32)[0]
            if np.isfinite(t) and t <= np.float32(2.0 ** 127):
                thr[i] = max(emin - int(scale_exp[i]) + 127, 1)
    layer = np.searchsorted(offs, np.arange(n), side="right") - 1
    return s, byte < thr[layer]


FORMATS = [F(5, 2), F(4, 3), F(3, 0), F(2, 1), F(5, 10), F(8, 7), F(6, 1), F(4, 3, 5), F(3, 2), F(2, 0)]


def _layout(sizes, pad=64):
    offs = np.zeros(len(sizes) + 1, np.int64)
    offs[1:] = np.cumsum(sizes)
    n = int(offs[-1])
    return offs, n, max(4, (n + pad - 1) // pad * pad)


def _check(G, n, offs, f, W):
    of = ofmt(f)
    mab = O.layer_maxabs(G, n, offs)
    se = O.layer_scales(mab, W, of)
    ref = O.sim_reduce(G, n, offs, se, of)
    s, flagged = model(G, n, offs, f, W, se, mab)
    ok = ~flagged
    a, b = s[ok].view(np.uint32), ref[ok].view(np.uint32)
    nan = np.isnan(s[ok]) & np.isnan(ref[ok])
    bad = (a != b) & ~nan
    assert not bad.any(), (str(f), W, np.nonzero(ok)[0][bad][:5])
    if f.m <= 7:
        low = ((a & np.uint32(0xFFFF)) != 0) & ~nan
        assert not low.any(), (str(f), W, "accepted sums with bits below 2^16", np.nonzero(ok)[0][low][:5])
    fa, fb = s[flagged], ref[flagged]
    differ = ~((fa.view(np.uint32) == fb.view(np.uint32)) | (np.isnan(fa) & np.isnan(fb)))
    return int(flagged.sum()), int(differ.sum())


@pytest.mark.parametrize("f", FORMATS, ids=str)
def test_accepted_elements_match_the_oracle(f):
    rng = np.random.default_rng(700 + 16 * f.e + f.m)
    offs, n, ld = _layout([1, 7, 900, 2, 1500, 64, 300, 33])
    n_flag = n_diff = 0
    for W in (1, 2, 4, 8, 64, 256):
        G = threshold_values(rng, W, ld, offs, f, LAYER_MAXIMA)
        a, b = _check(G, n, offs, f, W)
        n_flag += a
        n_diff += b
        # plain Gaussian layers with zeros, scales spread over 40 binades
        H = np.zeros((W, ld), np.float32)
        for i in range(offs.size - 1):
            lo, hi = offs[i], offs[i + 1]
            H[:, lo:hi] = rng.standard_normal((W, hi - lo)) * 2.0 ** rng.uniform(-30, 10)
        H[rng.random(H.shape) < 0.03] = 0
        a, b = _check(H, n, offs, f, W)
        n_flag += a
        n_diff += b
    assert n_flag > 0
    assert n_diff > 0, "the recomputed elements never differ: the criterion is not shown to matter"


@pytest.mark.parametrize("f", [F(5, 2), F(4, 3), F(2, 1)], ids=str)
def test_special_values_make_the_layer_recomputed(f):
    offs, n, ld = _layout([40, 40, 40, 40])
    G = np.full((4, ld), 0.5, np.float32)
    G[1, 3] = np.inf
    G[2, 45] = np.nan
    G[0, 80:120] = 3e38           # N * ghat overflows fp32
    G[3, 125] = 1e38              # N * ghat above 2^127
    G[:, n:] = 0
    mab = O.layer_maxabs(G, n, offs)
    se = O.layer_scales(mab, 4, ofmt(f))
    _, flagged = model(G, n, offs, f, 4, se, mab)
    assert flagged.all()


@pytest.mark.parametrize("f", [F(5, 2), F(4, 3), F(3, 0), F(5, 10), F(8, 7), F(3, 2)], ids=str)
@pytest.mark.parametrize("W", [1, 2, 4, 8, 16, 64, 256])
def test_worst_chain_stays_below_two_to_emax(f, W):
    """The no-overflow step of the claim: with every scaled input at the
    bound 2^emax / W, the rounded chain counts exactly to min(W, 2^(m+1))
    inputs (m = 0: 1, 2, 4, then stays) and stays, so its largest partial
    sum is 2^emax / W times that count, never above 2^emax."""
    emax, emin = (1 << f.e) - 2 - f.b, 1 - f.b
    c = 2.0 ** (emax - int(np.log2(W)))
    if c < 2.0 ** emin:
        pytest.skip("bound below the normal range")
    G = np.full((W, 4), c, np.float32)
    offs = np.array([0, 4], np.int64)
    out = O.sim_reduce(G, 4, offs, np.zeros(1, np.int32), ofmt(f), flags=O.OUTPUT_SCALED)
    cap = 4 if f.m == 0 else 2 ** (f.m + 1)
    assert np.all(out == np.float32(c * min(W, cap)))
    assert np.all(out <= 2.0 ** emax)
