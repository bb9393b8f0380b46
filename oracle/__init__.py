"""CPU oracle for the APS gradient path -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The HIP library never loads it and it
loads nothing of the HIP library.

The arithmetic lives in ``oracle.c`` (plain C99, exact double rounding; see its
header for the paper passages and the readings it follows).  This module only
builds that file with gcc and marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

INPUT_QUANTIZED = 1
OUTPUT_SCALED = 2
ACC_SEQUENTIAL = 0
ACC_KAHAN = 1


GCC_FLAGS = ["-std=c99", "-O2", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math", "-ffp-contract=off",
             "-Wall", "-Wextra"]


def build(force: bool = True, src: str = _SRC, out: str = _LIB) -> str:
    """Compile oracle.c into liboracle.so with gcc (IEEE semantics: no fast-math)."""
    if force or not os.path.exists(out):
        tmp = out + ".tmp"
        cmd = ["gcc", *GCC_FLAGS, "-I", _HERE, "-o", tmp, src, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return out


class _Fmt(ctypes.Structure):
    _fields_ = [("e", ctypes.c_int32), ("m", ctypes.c_int32), ("bias", ctypes.c_int32)]


@dataclass(frozen=True)
class Format:
    """A custom float (1 sign bit, e exponent bits, m mantissa bits, bias)."""

    e: int
    m: int
    bias: int | None = None

    @property
    def b(self) -> int:
        return (1 << (self.e - 1)) - 1 if self.bias is None else self.bias

    def c(self) -> _Fmt:
        return _Fmt(self.e, self.m, self.b)

    @property
    def bits(self) -> int:
        return 1 + self.e + self.m


_lib = None


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("APS_ORACLE_LIB")  # a mutated build, used by the pin-strength tests
        if path is None:
            path = _LIB
            if not os.path.exists(path):
                build(force=False)
        L = ctypes.CDLL(path)
        P = ctypes.c_void_p
        i32, i64, u32, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_double
        sig = {
            "oracle_format_ok": (ctypes.c_int, [_Fmt]),
            "oracle_emin": (ctypes.c_int, [_Fmt]),
            "oracle_emax": (ctypes.c_int, [_Fmt]),
            "oracle_maxfinite": (f64, [_Fmt]),
            "oracle_minsub": (f64, [_Fmt]),
            "oracle_round": (f64, [f64, _Fmt]),
            "oracle_ceil_log2": (ctypes.c_int, [f64]),
            "oracle_find_max_exp": (i32, [P, i64, i32, P]),
            "oracle_layer_maxabs": (None, [P, i32, i64, i64, P, i32, P]),
            "oracle_scale_one": (i32, [u32, i32, _Fmt]),
            "oracle_layer_scales": (None, [P, i32, i32, P, P, P]),
            "oracle_quantize": (None, [P, i32, i64, i64, P, i32, P, P, P, P]),
            "oracle_sim_reduce": (None, [P, i32, i64, i64, P, i32, P, P, P, u32, P]),
            "oracle_dequantize": (None, [P, P, i64, P, i32, P, P, P, P]),
            "oracle_encode": (u32, [f64, _Fmt]),
            "oracle_decode": (f64, [u32, _Fmt]),
            "oracle_pack_codes": (None, [P, i64, P, i32, P, P, P]),
            "oracle_sim_reduce_codes": (None, [P, i32, i64, i64, P, i32, P, P, P, u32, P]),
            "oracle_sim_reduce_ex": (None, [P, i32, i64, i64, P, i32, P, P, P, u32, i32, i32, P]),
            "oracle_round_off_error": (f64, [P, P, i64]),
            "oracle_lp_gemm": (None, [P, i64, P, i64, P, i64, i32, i32, i32, _Fmt, _Fmt, i32]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


# ------------------------------------------------------------ helpers

def _ptr(a: np.ndarray | None):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _fmts(fmts) -> ctypes.Array:
    if isinstance(fmts, Format):
        fmts = [fmts]
    arr = (_Fmt * len(fmts))()
    for k, f in enumerate(fmts):
        arr[k] = f.c()
    return arr


def _idx(fmt_idx):
    return None if fmt_idx is None else _c(fmt_idx, np.uint8)


# ------------------------------------------------------------ scalar API

def format_ok(f: Format) -> bool:
    return bool(lib().oracle_format_ok(f.c()))


def emin(f: Format) -> int:
    return lib().oracle_emin(f.c())


def emax(f: Format) -> int:
    return lib().oracle_emax(f.c())


def maxfinite(f: Format) -> float:
    return lib().oracle_maxfinite(f.c())


def minsub(f: Format) -> float:
    return lib().oracle_minsub(f.c())


def round_(y: float, f: Format) -> float:
    return lib().oracle_round(float(y), f.c())


def round_array(y: np.ndarray, f: Format) -> np.ndarray:
    fc = f.c()
    fn = lib().oracle_round
    flat = np.asarray(y, dtype=np.float64).ravel()
    return np.array([fn(float(v), fc) for v in flat], dtype=np.float64).reshape(np.shape(y))


def ceil_log2(t: float) -> int:
    return lib().oracle_ceil_log2(float(t))


def find_max_exp(g: np.ndarray, N: int):
    g = _c(g, np.float32)
    nf = ctypes.c_int32(0)
    r = lib().oracle_find_max_exp(_ptr(g), g.size, int(N), ctypes.byref(nf))
    return r, bool(nf.value)


def scale_one(maxabs_bits: int, N: int, f: Format) -> int:
    return lib().oracle_scale_one(ctypes.c_uint32(maxabs_bits), int(N), f.c())


def encode(v: float, f: Format) -> int:
    return lib().oracle_encode(float(v), f.c())


def decode(code: int, f: Format) -> float:
    return lib().oracle_decode(ctypes.c_uint32(code), f.c())


# ------------------------------------------------------------ array API
# G is a [W][ld] float32 array (worker-major); offsets is int64[L+1].

def layer_maxabs(G: np.ndarray, n: int, offsets: np.ndarray) -> np.ndarray:
    G = _c(G, np.float32)
    offs = _c(offsets, np.int64)
    L = offs.size - 1
    out = np.zeros(L, dtype=np.uint32)
    W, ld = G.shape
    lib().oracle_layer_maxabs(_ptr(G), W, ld, n, _ptr(offs), L, _ptr(out))
    return out


def layer_scales(maxabs_bits: np.ndarray, N: int, fmts, fmt_idx=None) -> np.ndarray:
    mb = _c(maxabs_bits, np.uint32)
    L = mb.size
    out = np.zeros(L, dtype=np.int32)
    idx = _idx(fmt_idx)
    lib().oracle_layer_scales(_ptr(mb), L, int(N), _fmts(fmts), _ptr(idx), _ptr(out))
    return out


def quantize(X: np.ndarray, n: int, offsets, scale_exp, fmts, fmt_idx=None) -> np.ndarray:
    X = _c(X, np.float32)
    offs = _c(offsets, np.int64)
    se = None if scale_exp is None else _c(scale_exp, np.int32)
    idx = _idx(fmt_idx)
    W, ld = X.shape
    Q = np.zeros_like(X)
    lib().oracle_quantize(_ptr(X), W, ld, n, _ptr(offs), offs.size - 1, _ptr(se),
                          _fmts(fmts), _ptr(idx), _ptr(Q))
    return Q


def sim_reduce(G: np.ndarray, n: int, offsets, scale_exp, fmts, fmt_idx=None,
               flags: int = 0) -> np.ndarray:
    G = _c(G, np.float32)
    offs = _c(offsets, np.int64)
    se = None if scale_exp is None else _c(scale_exp, np.int32)
    idx = _idx(fmt_idx)
    W, ld = G.shape
    out = np.zeros(n, dtype=np.float32)
    lib().oracle_sim_reduce(_ptr(G), W, ld, n, _ptr(offs), offs.size - 1, _ptr(se),
                            _fmts(fmts), _ptr(idx), int(flags), _ptr(out))
    return out


def code_bytes(n: int, bits: int) -> int:
    if bits <= 4:
        return (n + 1) // 2
    if bits <= 8:
        return n
    return 2 * n


def pack_codes(V: np.ndarray, offsets, fmts, fmt_idx=None) -> np.ndarray:
    V = _c(V, np.float32)
    offs = _c(offsets, np.int64)
    fl = [fmts] if isinstance(fmts, Format) else list(fmts)
    bits = max(f.bits for f in fl)
    out = np.zeros(code_bytes(V.size, bits), dtype=np.uint8)
    lib().oracle_pack_codes(_ptr(V), V.size, _ptr(offs), offs.size - 1, _fmts(fmts),
                            _ptr(_idx(fmt_idx)), _ptr(out))
    return out


def dequantize(Q, codes, n: int, offsets, scale_exp, fmts, fmt_idx=None) -> np.ndarray:
    offs = _c(offsets, np.int64)
    q = None if Q is None else _c(Q, np.float32)
    c = None if codes is None else _c(codes, np.uint8)
    se = None if scale_exp is None else _c(scale_exp, np.int32)
    out = np.zeros(n, dtype=np.float32)
    lib().oracle_dequantize(_ptr(q), _ptr(c), n, _ptr(offs), offs.size - 1, _ptr(se),
                            _fmts(fmts), _ptr(_idx(fmt_idx)), _ptr(out))
    return out


def sim_reduce_codes(codes: np.ndarray, W: int, ld: int, n: int, offsets, scale_exp, fmts, fmt_idx=None,
                     flags: int = 0) -> np.ndarray:
    """codes: uint8 array of W rows of packed codes, row stride ld elements."""
    c = _c(codes, np.uint8)
    offs = _c(offsets, np.int64)
    se = None if scale_exp is None else _c(scale_exp, np.int32)
    out = np.zeros(n, dtype=np.float32)
    lib().oracle_sim_reduce_codes(_ptr(c), int(W), int(ld), int(n), _ptr(offs), offs.size - 1, _ptr(se),
                                  _fmts(fmts), _ptr(_idx(fmt_idx)), int(flags), _ptr(out))
    return out


def sim_reduce_ex(G: np.ndarray, n: int, offsets, scale_exp, fmts, fmt_idx=None, flags: int = 0,
                  group: int | None = None, accumulator: int = ACC_SEQUENTIAL) -> np.ndarray:
    G = _c(G, np.float32)
    offs = _c(offsets, np.int64)
    se = None if scale_exp is None else _c(scale_exp, np.int32)
    W, ld = G.shape
    k = W if group is None else int(group)
    out = np.zeros(n, dtype=np.float32)
    lib().oracle_sim_reduce_ex(_ptr(G), W, ld, n, _ptr(offs), offs.size - 1, _ptr(se), _fmts(fmts),
                               _ptr(_idx(fmt_idx)), int(flags), k, int(accumulator), _ptr(out))
    return out


def round_off_error(grad_h: np.ndarray, grad_l: np.ndarray) -> float:
    h = _c(grad_h, np.float32)
    l = _c(grad_l, np.float32)
    return lib().oracle_round_off_error(_ptr(h), _ptr(l), h.size)


def lp_gemm(A: np.ndarray, B: np.ndarray, fin: Format, facc: Format, accumulator: int = ACC_SEQUENTIAL) -> np.ndarray:
    """C = A @ B on a low-precision multiply-accumulate unit (A: [M][K], B: [K][N])."""
    A = _c(A, np.float32)
    B = _c(B, np.float32)
    M, K = A.shape
    K2, N = B.shape
    assert K == K2
    C = np.zeros((M, N), dtype=np.float32)
    lib().oracle_lp_gemm(_ptr(A), max(K, 1), _ptr(B), max(N, 1), _ptr(C), max(N, 1), M, N, K,
                         fin.c(), facc.c(), int(accumulator))
    return C
