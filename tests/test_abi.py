"""Host-side checks of the C ABI: the library loads, exports what the header
declares, and rejects bad arguments before anything is enqueued.

Every call below carries at least one invalid argument, so none of them ever
reaches a kernel launch (these tests run without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_1911_08907_amd import aps as A
from paper_1911_08907_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "aps.h")


def _gpu_visible() -> bool:
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:
        return False


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(A.LIB_PATH):
        B.build()
    return A.lib()


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(aps_[a-z_]+)\s*\(", txt)))


def test_header_declares_the_five_calls():
    d = _declared()
    for name in ("aps_layer_maxabs", "aps_layer_scales", "aps_quantize", "aps_sim_reduce", "aps_dequantize",
                 "aps_sim_reduce_codes", "aps_sim_reduce_ex"):
        assert name in d


def test_every_declared_symbol_is_exported(lib):
    for name in _declared():
        assert hasattr(lib, name), name
    assert set(_declared()) == set(A.EXPORTS)


def test_strerror(lib):
    for st in (0, -1, -2, -3, -4, -5, -6):
        assert A.strerror(st) and A.strerror(st) != "unknown status"
    assert A.strerror(12345) == "unknown status"


@pytest.mark.parametrize("f,ok", [
    (A.Format(5, 2), A.APS_OK), (A.Format(4, 3), A.APS_OK), (A.Format(3, 0), A.APS_OK),
    (A.Format(2, 0), A.APS_OK), (A.Format(8, 23), A.APS_OK), (A.Format(8, 7), A.APS_OK),
    (A.Format(8, 0), A.APS_OK), (A.Format(5, 10), A.APS_OK), (A.Format(6, 9), A.APS_OK),
    (A.Format(7, 23), A.APS_OK), (A.Format(4, 3, 5), A.APS_OK), (A.Format(5, 2, 20), A.APS_OK),
    (A.Format(1, 2), A.APS_ERR_FORMAT), (A.Format(9, 2), A.APS_ERR_FORMAT),
    (A.Format(5, 24), A.APS_ERR_FORMAT), (A.Format(5, -1), A.APS_ERR_FORMAT),
    (A.Format(8, 7, 126), A.APS_ERR_FORMAT),      # emax 128
    (A.Format(8, 7, 128), A.APS_OK),               # e = 8, another bias: rounded in fp64
    (A.Format(7, 20, 127), A.APS_OK),              # subnormals below 2^-126: rounded in fp64
    (A.Format(5, 2, 200), A.APS_ERR_FORMAT),       # smallest subnormal below 2^-149
])
def test_format_supported(lib, f, ok):
    assert A.format_supported(f) == ok


def _pal(*fs):
    arr = (A.aps_format * max(1, len(fs)))()
    for i, f in enumerate(fs):
        arr[i] = f.c()
    return arr


# The calls below pass fake device pointers; each also carries an invalid
# argument so validation rejects it first.  They are skipped where a GPU is
# visible, so that a wrong expectation can never turn into a launch.
no_gpu = pytest.mark.skipif(_gpu_visible(), reason="host-validation tests use fake pointers")

P = ctypes.c_void_p
GOOD = P(4096)      # an aligned non-NULL value; never dereferenced by these calls
MIS = P(4100)       # misaligned


@no_gpu
def test_maxabs_validation(lib):
    f = lib.aps_layer_maxabs
    assert f(None, 2, 64, 64, GOOD, 1, GOOD, None) == A.APS_ERR_NULL
    assert f(GOOD, 2, 64, 64, None, 1, GOOD, None) == A.APS_ERR_NULL
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, None) == A.APS_ERR_NULL
    assert f(GOOD, 0, 64, 64, GOOD, 1, GOOD, None) == A.APS_ERR_SIZE
    assert f(GOOD, (1 << 24) + 1, 64, 64, GOOD, 1, GOOD, None) == A.APS_ERR_SIZE
    assert f(GOOD, 2, 64, 64, GOOD, 0, GOOD, None) == A.APS_ERR_SIZE
    assert f(GOOD, 2, 60, 64, GOOD, 1, GOOD, None) == A.APS_ERR_SIZE     # ld < n
    assert f(GOOD, 2, 64, -1, GOOD, 1, GOOD, None) == A.APS_ERR_SIZE
    assert f(GOOD, 2, 66, 64, GOOD, 1, GOOD, None) == A.APS_ERR_ALIGN    # ld % 4
    assert f(MIS, 2, 64, 64, GOOD, 1, GOOD, None) == A.APS_ERR_ALIGN


@no_gpu
def test_scales_validation(lib):
    f = lib.aps_layer_scales
    pal = _pal(A.Format(5, 2))
    assert f(None, 4, 8, pal, 1, None, GOOD, None) == A.APS_ERR_NULL
    assert f(GOOD, 4, 8, pal, 1, None, None, None) == A.APS_ERR_NULL
    assert f(GOOD, 4, 8, None, 1, None, GOOD, None) == A.APS_ERR_NULL
    assert f(GOOD, 0, 8, pal, 1, None, GOOD, None) == A.APS_ERR_SIZE
    assert f(GOOD, 4, 0, pal, 1, None, GOOD, None) == A.APS_ERR_SIZE
    assert f(GOOD, 4, 8, pal, 0, None, GOOD, None) == A.APS_ERR_SIZE
    assert f(GOOD, 4, 8, _pal(*[A.Format(5, 2)] * 9), 9, None, GOOD, None) == A.APS_ERR_SIZE
    assert f(GOOD, 4, 8, _pal(A.Format(9, 2)), 1, None, GOOD, None) == A.APS_ERR_FORMAT
    assert f(GOOD, 4, 8, _pal(A.Format(5, 2), A.Format(8, 3, 100)), 2, None, GOOD, None) == A.APS_ERR_FORMAT


@no_gpu
def test_quantize_validation(lib):
    f = lib.aps_quantize
    pal = _pal(A.Format(5, 2))
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, pal, 1, None, None, None, None) == A.APS_ERR_NULL
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, pal, 1, None, MIS, None, None) == A.APS_ERR_ALIGN
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, pal, 1, None, None, MIS, None) == A.APS_ERR_ALIGN
    # codes need one container class across the palette, and at most 16 bits
    two = _pal(A.Format(5, 2), A.Format(5, 10))
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, two, 2, None, None, GOOD, None) == A.APS_ERR_UNSUPPORTED
    wide = _pal(A.Format(8, 23))
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, wide, 1, None, None, GOOD, None) == A.APS_ERR_UNSUPPORTED
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, _pal(A.Format(5, 30)), 1, None, GOOD, None, None) == A.APS_ERR_FORMAT


@no_gpu
def test_sim_reduce_validation(lib):
    f = lib.aps_sim_reduce
    pal = _pal(A.Format(5, 2))
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, pal, 1, None, 0, None, None, None) == A.APS_ERR_NULL
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, pal, 1, None, 0, MIS, None, None) == A.APS_ERR_ALIGN
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, pal, 1, None, 4, GOOD, None, None) == A.APS_ERR_UNSUPPORTED
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, _pal(A.Format(9, 2)), 1, None, 0, GOOD, None,
             None) == A.APS_ERR_FORMAT
    assert f(None, 2, 64, 64, GOOD, 1, None, pal, 1, None, 0, GOOD, None, None) == A.APS_ERR_NULL


@no_gpu
def test_dequantize_validation(lib):
    f = lib.aps_dequantize
    pal = _pal(A.Format(5, 2))
    assert f(None, None, 64, GOOD, 1, None, pal, 1, None, GOOD, None) == A.APS_ERR_NULL
    assert f(GOOD, None, 64, GOOD, 1, None, pal, 1, None, None, None) == A.APS_ERR_NULL
    assert f(GOOD, None, 64, GOOD, 0, None, pal, 1, None, GOOD, None) == A.APS_ERR_SIZE
    assert f(GOOD, None, 64, GOOD, 1, None, pal, 1, None, MIS, None) == A.APS_ERR_ALIGN
    assert f(None, GOOD, 64, GOOD, 1, None, _pal(A.Format(8, 23)), 1, None, GOOD, None) == A.APS_ERR_UNSUPPORTED


@no_gpu
def test_sim_reduce_codes_validation(lib):
    f = lib.aps_sim_reduce_codes
    pal = _pal(A.Format(5, 2))
    assert f(None, 2, 64, 64, GOOD, 1, None, pal, 1, None, 0, GOOD, None, None) == A.APS_ERR_NULL
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, pal, 1, None, 0, None, None, None) == A.APS_ERR_NULL
    assert f(GOOD, 0, 64, 64, GOOD, 1, None, pal, 1, None, 0, GOOD, None, None) == A.APS_ERR_SIZE
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, pal, 1, None, 1, GOOD, None, None) == A.APS_ERR_UNSUPPORTED
    assert f(MIS, 2, 64, 64, GOOD, 1, None, pal, 1, None, 0, GOOD, None, None) == A.APS_ERR_ALIGN
    assert f(GOOD, 2, 68, 64, GOOD, 1, None, pal, 1, None, 0, GOOD, None, None) == A.APS_ERR_ALIGN   # 68-byte rows
    assert f(GOOD, 2, 64, 64, GOOD, 1, None, _pal(A.Format(8, 23)), 1, None, 0, GOOD, None,
             None) == A.APS_ERR_UNSUPPORTED


@no_gpu
def test_sim_reduce_ex_validation(lib):
    f = lib.aps_sim_reduce_ex
    pal = _pal(A.Format(5, 2))
    o = lambda k, acc: ctypes.byref(A.aps_reduce_opts(k, acc))
    assert f(GOOD, 8, 64, 64, GOOD, 1, None, pal, 1, None, 0, o(3, 0), GOOD, None, None) == A.APS_ERR_SIZE
    assert f(GOOD, 8, 64, 64, GOOD, 1, None, pal, 1, None, 0, o(16, 0), GOOD, None, None) == A.APS_ERR_SIZE
    assert f(GOOD, 8, 64, 64, GOOD, 1, None, pal, 1, None, 0, o(0, 0), GOOD, None, None) == A.APS_ERR_SIZE
    assert f(GOOD, 8, 64, 64, GOOD, 1, None, pal, 1, None, 0, o(2, 7), GOOD, None, None) == A.APS_ERR_UNSUPPORTED
    assert f(None, 8, 64, 64, GOOD, 1, None, pal, 1, None, 0, o(2, 1), GOOD, None, None) == A.APS_ERR_NULL
    assert f(GOOD, 8, 64, 64, GOOD, 1, None, pal, 1, None, 0, o(2, 1), None, None, None) == A.APS_ERR_NULL
    assert f(GOOD, 8, 64, 64, GOOD, 1, None, pal, 1, None, 0, o(2, 1), MIS, None, None) == A.APS_ERR_ALIGN


@no_gpu
def test_lp_gemm_validation(lib):
    f = lib.aps_lp_gemm
    F5, F8 = A.Format(5, 2).c(), A.Format(8, 23).c()
    g = lambda M=8, N=8, K=8, lda=8, ldb=8, ldc=8, a=GOOD, b=GOOD, c=GOOD, fin=F5, facc=F5, acc=0: \
        f(a, lda, b, ldb, c, ldc, M, N, K, fin, facc, acc, None)
    assert g(M=-1) == A.APS_ERR_SIZE
    assert g(K=(1 << 22) + 1, lda=1 << 23) == A.APS_ERR_SIZE
    assert g(c=None) == A.APS_ERR_NULL
    assert g(a=None) == A.APS_ERR_NULL
    assert g(lda=7) == A.APS_ERR_SIZE
    assert g(ldb=7) == A.APS_ERR_SIZE
    assert g(ldc=7) == A.APS_ERR_SIZE
    assert g(fin=A.aps_format(9, 2, 255)) == A.APS_ERR_FORMAT
    assert g(acc=5) == A.APS_ERR_UNSUPPORTED
    # products of two 13-bit significands are not exact in fp32
    assert g(fin=A.Format(5, 12).c()) == A.APS_ERR_UNSUPPORTED
    # bf16-range inputs with 12-bit significands: tiny products would need
    # fp32's subnormal rounding, which the fp32 accumulator format can see
    assert g(fin=A.Format(8, 11).c(), facc=F8) == A.APS_ERR_UNSUPPORTED
    # formats rounded in fp64 are not built into the GEMM, as input or accumulator
    assert g(fin=A.Format(5, 10, 120).c()) == A.APS_ERR_UNSUPPORTED
    assert g(facc=A.Format(8, 7, 130).c()) == A.APS_ERR_UNSUPPORTED
    # empty output: nothing to do (and nothing checked beyond the sizes)
    assert g(M=0, a=None, b=None, c=None) == A.APS_OK


def test_sync_workspace_bytes(lib):
    f = A.aps_sync_workspace_bytes
    up = lambda b: (b + 255) // 256 * 256
    for n, L in ((0, 1), (1, 1), (1024, 64), (1025, 65), (25557032, 161), (335141888, 391)):
        C = (n + 1023) // 1024
        assert f(n, L) == up(1024 * C) + up(4 * C) + up(4 * L) + 256 + up(4 * C) + 2048 * C + up(4 * L) + up(C), (n, L)
    assert f(-1, 3) == 0 and f(5, -1) == 0 and f((1 << 30) + 1, 1) == 0


@no_gpu
def test_sync_validation(lib):
    f = lib.aps_sync
    pal = _pal(A.Format(5, 2))
    ws = A.aps_sync_workspace_bytes(64, 1)
    ok = dict(G=GOOD, W=2, ld=64, n=64, off=GOOD, L=1, pal=pal, nf=1, idx=None, ph=3, mab=GOOD, se=GOOD,
              out=GOOD, ws=GOOD, wsb=ws)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["G"], a["W"], a["ld"], a["n"], a["off"], a["L"], a["pal"], a["nf"], a["idx"], a["ph"],
                 a["mab"], a["se"], a["out"], a["ws"], a["wsb"], None)

    assert call(G=None, ph=0) == A.APS_ERR_NULL
    assert call(mab=None) == A.APS_ERR_NULL
    assert call(se=None) == A.APS_ERR_NULL
    assert call(out=None) == A.APS_ERR_NULL
    assert call(ws=None) == A.APS_ERR_NULL
    assert call(ph=0) == A.APS_ERR_UNSUPPORTED
    assert call(ph=4) == A.APS_ERR_UNSUPPORTED                  # a route but no pass
    assert call(ph=32 | 3) == A.APS_ERR_UNSUPPORTED             # unknown bit
    assert call(ph=3 | 4 | 8) == A.APS_ERR_UNSUPPORTED          # two routes
    assert call(ph=3 | 4 | 16) == A.APS_ERR_UNSUPPORTED
    assert call(ph=3 | 8 | 16) == A.APS_ERR_UNSUPPORTED
    assert call(out=MIS) == A.APS_ERR_ALIGN
    assert call(ws=P(4096 + 128)) == A.APS_ERR_ALIGN       # workspace needs 256-byte alignment
    assert call(wsb=ws - 1) == A.APS_ERR_SIZE
    assert call(W=0) == A.APS_ERR_SIZE
    assert call(W=(1 << 24) + 1) == A.APS_ERR_SIZE
    assert call(n=(1 << 30) + 4, ld=(1 << 30) + 4) == A.APS_ERR_SIZE   # above APS_MAX_ELEMS
    assert call(pal=_pal(A.Format(9, 2))) == A.APS_ERR_FORMAT
    assert call(nf=0) == A.APS_ERR_SIZE


def test_sync_route_choice(lib):
    F = A.Format
    one, two, guess = A.APS_SYNC_ONE_PASS, A.APS_SYNC_TWO_PASS, A.APS_SYNC_GUESS
    ONE, TWO, GUESS = A.APS_SYNC_ROUTE_ONE_PASS, A.APS_SYNC_ROUTE_TWO_PASS, A.APS_SYNC_ROUTE_GUESS
    r = A.aps_sync_route
    big, small = 25557032, 272474          # ResNet-50 and ResNet-20 element counts
    # the default takes one pass when the format's range leaves few elements to recompute
    assert r(256, big, [F(5, 2)]) == ONE
    assert r(8, small, [F(5, 2)]) == ONE
    assert r(8, big, [F(5, 10), F(5, 2)]) == ONE
    assert r(256, big, [F(8, 7)]) == ONE
    # otherwise the guessed-scale route for at least 2^26 element-workers, else two passes
    assert r(256, big, [F(4, 3)]) == GUESS
    assert r(256, (1 << 18) - 1, [F(4, 3)]) == TWO
    assert r(256, 1 << 18, [F(4, 3)]) == GUESS
    assert r(8, small, [F(3, 0)]) == TWO
    assert r(8, small, [F(4, 3)]) == TWO
    assert r(12, big, [F(5, 2)]) == GUESS        # W not a power of two
    assert r(8, big, [F(5, 12)]) == GUESS        # m > 10
    assert r(12, small, [F(5, 2)]) == TWO
    # forced routes; the one-pass route needs a power-of-two W and m <= 10
    assert r(256, big, [F(4, 3)], one) == ONE
    assert r(256, big, [F(5, 2)], two) == TWO
    assert r(256, big, [F(5, 2)], guess) == GUESS
    assert r(3, 1, [F(5, 12)], guess) == GUESS
    assert r(12, big, [F(5, 2)], one) == TWO
    # formats rounded in fp64 never take the one-pass route
    assert r(8, big, [F(8, 7, 130)]) == GUESS
    assert r(8, big, [F(5, 2), F(5, 10, 120)], one) == TWO
    assert r(8, big, [F(5, 12)], one) == TWO
    assert r(8, big, [F(5, 2), F(8, 23)], one) == TWO
    for bad in (one | two, one | guess, two | guess):
        with pytest.raises(A.ApsError):
            r(8, big, [F(5, 2)], bad)
    with pytest.raises(A.ApsError):
        r(0, big, [F(5, 2)])
    with pytest.raises(A.ApsError):
        r(8, -1, [F(5, 2)])
    with pytest.raises(A.ApsError):
        r(8, (1 << 30) + 1, [F(5, 2)])
    with pytest.raises(A.ApsError):
        r(8, big, [F(9, 2)])


@no_gpu
def test_sync_noalloc_validation(lib):
    """aps_sync_noalloc checks what aps_sync checks, then the set's
    workspace against its static array, all before touching the device."""
    f = lib.aps_sync_noalloc
    pal = _pal(A.Format(5, 2))
    ok = dict(G=GOOD, W=2, ld=64, n=64, off=GOOD, L=1, pal=pal, nf=1, idx=None, ph=3, mab=GOOD, se=GOOD,
              out=GOOD)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["G"], a["W"], a["ld"], a["n"], a["off"], a["L"], a["pal"], a["nf"], a["idx"], a["ph"],
                 a["mab"], a["se"], a["out"], None)

    assert call(G=None) == A.APS_ERR_NULL
    assert call(off=None) == A.APS_ERR_NULL
    assert call(mab=None) == A.APS_ERR_NULL
    assert call(se=None) == A.APS_ERR_NULL
    assert call(out=None) == A.APS_ERR_NULL
    assert call(W=0) == A.APS_ERR_SIZE
    assert call(n=65) == A.APS_ERR_SIZE                       # ld < n
    assert call(G=MIS) == A.APS_ERR_ALIGN
    # the largest n whose workspace fits the array, and the next chunk's worth
    limit = A.APS_SYNC_SCRATCH_BYTES
    n_fit = max(c * 1024 for c in range(1, 40000) if A.aps_sync_workspace_bytes(c * 1024, 1) <= limit)
    assert A.aps_sync_workspace_bytes(n_fit + 1, 1) > limit
    assert 25557032 <= n_fit < (1 << 30)                      # a ResNet-50's gradient fits
    assert call(n=n_fit + 1, ld=n_fit + 4) == A.APS_ERR_SIZE
    assert call(n=1 << 30, ld=1 << 30) == A.APS_ERR_SIZE
    big_L = 1 << 24                                            # many layers need more thresholds
    assert A.aps_sync_workspace_bytes(n_fit, big_L) > limit
    assert call(n=n_fit, ld=n_fit, L=big_L) == A.APS_ERR_SIZE
