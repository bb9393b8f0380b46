"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bit-exact comparison on every output (fp32 values bitwise, NaN as a class;
codes byte for byte), on seeded synthetic inputs: edge layouts, every code of
the small formats, the paper-shaped configurations (full where the oracle
finishes in seconds, sampled outputs otherwise)."""
import math
import time
import zlib

import numpy as np
import pytest
import torch

import oracle as O
from paper_1911_08907_amd import aps as A
from paper_1911_08907_amd import workloads as WL
from tests import exact_ref as X
from tests._util import first_diff, log, ofmt, same_f32, same_maxabs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    A.lib()  # the HIP library must be there: no fallback
    return torch.device("cuda:0")


def _code_cls(bits):
    return 0 if bits <= 4 else (1 if bits <= 8 else 2)


def _unpack(c: np.ndarray, n: int, bits: int) -> np.ndarray:
    cls = _code_cls(bits)
    if cls == 0:
        b = c[:(n + 1) // 2].astype(np.uint32)
        return np.stack([b & 15, b >> 4], 1).ravel()[:n]
    if cls == 1:
        return c[:n].astype(np.uint32)
    return c[:2 * n].view(np.uint16).astype(np.uint32)


def _codes_equal(g: np.ndarray, o: np.ndarray, n: int, bits: int, nan_mask=None) -> bool:
    """Compare packed code arrays over the first n elements only.  Where the
    value is NaN the sign bit of the code is unspecified and not compared."""
    if nan_mask is not None and nan_mask.any():
        gu, ou = _unpack(g, n, bits), _unpack(o, n, bits)
        keep = np.uint32((1 << (bits - 1)) - 1)
        gu = np.where(nan_mask, gu & keep, gu)
        ou = np.where(nan_mask, ou & keep, ou)
        return np.array_equal(gu, ou)
    cls = _code_cls(bits)
    if cls == 0:
        full = n // 2
        if not np.array_equal(g[:full], o[:full]):
            return False
        if n % 2:
            return (g[full] & 15) == (o[full] & 15)
        return True
    nb = n if cls == 1 else 2 * n
    return np.array_equal(g[:nb], o[:nb])


def _row_code_bytes(ld, bits):
    cls = _code_cls(bits)
    return ld // 2 if cls == 0 else (ld if cls == 1 else 2 * ld)


def run_case(dev, G: np.ndarray, n: int, offs: np.ndarray, pal, fmt_idx=None, mode="aps", N=None,
             scale_exp=None, codes=True, tag=""):
    """Run every entry point on the GPU and the oracle on the same bytes."""
    W, ld = G.shape
    L = offs.size - 1
    opal = [ofmt(f) for f in pal]
    G_t = torch.from_numpy(G).to(dev)
    offs_t = torch.from_numpy(offs).to(dev)
    idx_t = None if fmt_idx is None else torch.from_numpy(fmt_idx).to(dev)
    bits = {f.bits for f in pal}
    classes = {_code_cls(b) for b in bits}
    with_codes = codes and len(classes) == 1 and max(bits) <= 16
    cbits = max(bits)

    # max-abs (always) and scales (APS mode)
    mab = torch.zeros(L, dtype=torch.int32, device=dev)
    A.aps_layer_maxabs(G_t, n, offs_t, mab)
    o_mab = O.layer_maxabs(G, n, offs)
    torch.cuda.synchronize()
    assert same_maxabs(mab.cpu().numpy(), o_mab), f"{tag} maxabs"
    if mode == "aps":
        Nw = W if N is None else N
        se_t = torch.zeros(L, dtype=torch.int32, device=dev)
        A.aps_layer_scales(mab, Nw, pal, idx_t, se_t)
        o_se = O.layer_scales(o_mab, Nw, opal, fmt_idx)
        assert np.array_equal(se_t.cpu().numpy(), o_se), f"{tag} scales"
    elif mode == "raw":
        se_t, o_se = None, None
    else:  # explicit exponents
        o_se = np.asarray(scale_exp, np.int32)
        se_t = torch.from_numpy(o_se).to(dev)

    # quantize
    Q_t = torch.zeros_like(G_t)
    qc_t = torch.zeros(max(1, W * _row_code_bytes(ld, cbits)), dtype=torch.uint8, device=dev) if with_codes else None
    A.aps_quantize(G_t, n, offs_t, se_t, pal, idx_t, Q=Q_t, codes=qc_t)
    o_Q = O.quantize(G, n, offs, o_se, opal, fmt_idx)
    Qg = Q_t.cpu().numpy()
    ok = same_f32(Qg[:, :n], o_Q[:, :n])
    assert ok, f"{tag} quantize {first_diff(Qg[:, :n], o_Q[:, :n])}"
    if with_codes:
        qc = qc_t.cpu().numpy()
        rb = _row_code_bytes(ld, cbits)
        for w in range(W):
            oc = O.pack_codes(o_Q[w, :n], offs, opal, fmt_idx)
            assert _codes_equal(qc[w * rb:(w + 1) * rb], oc, n, cbits, np.isnan(o_Q[w, :n])), \
                f"{tag} quantize codes row {w}"

    # reduce of the quantized codes (the exchanged form), when rows are 16-byte aligned
    if with_codes and _row_code_bytes(ld, cbits) % 16 == 0 and n > 0:
        rc2 = torch.zeros(max(16, A.code_bytes(n, cbits)), dtype=torch.uint8, device=dev)
        o2 = torch.zeros(max(n, 1), dtype=torch.float32, device=dev)
        A.aps_sim_reduce_codes(qc_t, W, ld, n, offs_t, se_t, pal, idx_t, 0, out=o2, codes_out=rc2)
        oq = O.sim_reduce_codes(qc.reshape(W, -1), W, ld, n, offs, o_se, opal, fmt_idx)
        g2 = o2.cpu().numpy()[:n]
        assert same_f32(g2, oq), f"{tag} sim_reduce_codes {first_diff(g2, oq)}"
        oq_s = O.sim_reduce_codes(qc.reshape(W, -1), W, ld, n, offs, o_se, opal, fmt_idx, flags=O.OUTPUT_SCALED)
        assert _codes_equal(rc2.cpu().numpy(), O.pack_codes(oq_s, offs, opal, fmt_idx), n, cbits,
                            np.isnan(oq_s)), f"{tag} sim_reduce_codes codes"

    # fused reduce, plain and scaled output, with codes
    out_t = torch.zeros(max(n, 1), dtype=torch.float32, device=dev)
    rc_t = torch.zeros(max(16, A.code_bytes(n, cbits)), dtype=torch.uint8, device=dev) if with_codes else None
    A.aps_sim_reduce(G_t, n, offs_t, se_t, pal, idx_t, 0, out=out_t, codes_out=rc_t)
    o_out = O.sim_reduce(G, n, offs, o_se, opal, fmt_idx)
    og = out_t.cpu().numpy()[:n]
    assert same_f32(og, o_out), f"{tag} sim_reduce {first_diff(og, o_out)}"
    o_sc = O.sim_reduce(G, n, offs, o_se, opal, fmt_idx, flags=O.OUTPUT_SCALED)
    if with_codes:
        oc = O.pack_codes(o_sc, offs, opal, fmt_idx)
        assert _codes_equal(rc_t.cpu().numpy(), oc, n, cbits, np.isnan(o_sc)), f"{tag} sim_reduce codes"

    # composition: reduce of the quantized input, scaled output, then dequantize
    sc_t = torch.zeros(max(n, 1), dtype=torch.float32, device=dev)
    A.aps_sim_reduce(Q_t, n, offs_t, se_t, pal, idx_t, A.APS_INPUT_QUANTIZED | A.APS_OUTPUT_SCALED, out=sc_t)
    sg = sc_t.cpu().numpy()[:n]
    o_sc2 = O.sim_reduce(o_Q, n, offs, o_se, opal, fmt_idx, flags=O.INPUT_QUANTIZED | O.OUTPUT_SCALED)
    assert same_f32(sg, o_sc2), f"{tag} reduce(IN_Q|OUT_SCALED) {first_diff(sg, o_sc2)}"
    assert same_f32(o_sc2, o_sc), f"{tag} oracle composition"
    dq_t = torch.zeros(max(n, 1), dtype=torch.float32, device=dev)
    A.aps_dequantize(sc_t, None, n, offs_t, se_t, pal, idx_t, dq_t)
    dg = dq_t.cpu().numpy()[:n]
    assert same_f32(dg, o_out), f"{tag} dequantize(Q) {first_diff(dg, o_out)}"
    if with_codes:
        dq2_t = torch.zeros(max(n, 1), dtype=torch.float32, device=dev)
        A.aps_dequantize(None, rc_t, n, offs_t, se_t, pal, idx_t, dq2_t)
        d2 = dq2_t.cpu().numpy()[:n]
        # decode the same code bytes on both sides
        o_d2 = O.dequantize(None, rc_t.cpu().numpy(), n, offs, o_se, opal, fmt_idx)
        assert same_f32(d2, o_d2), f"{tag} dequantize(codes) {first_diff(d2, o_d2)}"
    return og


# ----------------------------------------------------------- edge layouts

F = A.Format
ALL_FORMATS = [F(5, 2), F(4, 3), F(3, 0), F(2, 0), F(2, 1), F(3, 2), F(5, 10), F(6, 9), F(8, 7), F(8, 23),
               F(8, 0), F(8, 15), F(5, 12), F(7, 23), F(4, 3, 5), F(5, 2, 20), F(6, 1), F(7, 5), F(2, 23),
               F(3, 12), F(2, 15)]  # the last two: LOW class with fp64 adds
# formats rounded in fp64: e = 8 with a bias other than 127, or a subnormal
# grid that reaches below 2^-126 (the scaled input is fl32, rounded by fp32's
# own underflow there)
GEN_FORMATS = [F(8, 7, 130), F(8, 0, 140), F(8, 20, 128), F(7, 20, 127), F(5, 10, 120), F(4, 3, 140),
               F(3, 0, 145), F(2, 1, 147)]
ALL_FORMATS += GEN_FORMATS

SIZES = [0, 1, 3, 5, 7, 1023, 1024, 1025, 2049, 0, 64, 13, 4095, 2, 3000]


def _layout(sizes, pad_to=64):
    offs = np.zeros(len(sizes) + 1, np.int64)
    offs[1:] = np.cumsum(sizes)
    n = int(offs[-1])
    ld = max(4, (n + pad_to - 1) // pad_to * pad_to)
    return offs, n, ld


def _values(rng, W, ld, offs, kind):
    L = offs.size - 1
    G = np.zeros((W, ld), np.float32)
    for i in range(L):
        a, b = offs[i], offs[i + 1]
        if b == a:
            continue
        s = 2.0 ** rng.uniform(-40, 10) if kind != "tiny" else 2.0 ** rng.uniform(-149, -100)
        G[:, a:b] = (rng.standard_normal((W, b - a)) * s).astype(np.float32)
        r = rng.random((W, b - a))
        G[:, a:b][r < 0.05] = 0.0
        G[:, a:b][(r >= 0.05) & (r < 0.07)] = -0.0
    if kind == "special":
        flat = G[:, :offs[-1]]
        k = flat.size
        for val, cnt in ((np.nan, 3), (np.inf, 3), (-np.inf, 3), (3e38, 5), (1e-45, 5), (-1e-40, 5)):
            idx = rng.integers(0, k, cnt)
            flat.reshape(-1)[idx] = val
    # padding past n holds garbage that must not matter
    G[:, offs[-1]:] = np.nan
    return G


@pytest.mark.parametrize("f", ALL_FORMATS, ids=str)
@pytest.mark.parametrize("kind", ["normal", "special", "tiny"])
def test_edge_layouts_single_format(dev, f, kind):
    seed = zlib.crc32(f"{f}/{kind}".encode())  # stable across interpreters
    rng = np.random.default_rng(seed)
    offs, n, ld = _layout(SIZES)
    for W in (1, 2, 3, 8, 13):
        G = _values(rng, W, ld, offs, kind)
        tag = f"{f} {kind} W={W} seed={seed}"
        log("case", tag)
        run_case(dev, G, n, offs, [f], mode="aps", tag=tag + " aps")
        run_case(dev, G, n, offs, [f], mode="raw", tag=tag + " raw")
        se = rng.integers(-300, 300, offs.size - 1).astype(np.int32)
        run_case(dev, G, n, offs, [f], mode="exp", scale_exp=se, tag=tag + " exp")
    # N different from W (non power of two)
    G = _values(rng, 5, ld, offs, kind)
    run_case(dev, G, n, offs, [f], mode="aps", N=7, tag=f"{f} {kind} W=5 N=7")


@pytest.mark.parametrize("seed", range(6))
def test_edge_layouts_mixed_palette(dev, seed):
    rng = np.random.default_rng(100 + seed)
    pal_choices = [[F(5, 2), F(4, 3), F(3, 0), F(2, 1)],        # 4-8 bit codes mix classes
                   [F(5, 2), F(4, 3), F(6, 1), F(3, 4)],         # all byte codes
                   [F(5, 10), F(5, 2), F(8, 7)],
                   [F(8, 23), F(5, 12), F(3, 0), F(8, 0), F(4, 3, 5)]]
    pal = pal_choices[seed % len(pal_choices)]
    sizes = [int(v) for v in rng.choice([0, 1, 2, 3, 5, 17, 255, 1000, 1023, 1024, 1500, 4096], 40)]
    offs, n, ld = _layout(sizes)
    fmt_idx = rng.integers(0, len(pal), len(sizes)).astype(np.uint8)
    for W in (1, 4, 9):
        G = _values(rng, W, ld, offs, "special" if seed % 2 else "normal")
        tag = f"mixed seed={seed} W={W}"
        log("case", tag)
        run_case(dev, G, n, offs, pal, fmt_idx=fmt_idx, mode="aps", tag=tag + " aps")
        run_case(dev, G, n, offs, pal, fmt_idx=fmt_idx, mode="raw", tag=tag + " raw")


def test_quantize_mixed_palette_many_workers(dev):
    """A two-format palette at W = 2^17 workers (more than a grid's y extent
    of 65535 blocks) on a tiny gradient: values and 8-bit codes of every row,
    in APS and RAW mode."""
    rng = np.random.default_rng(4217)
    W = 1 << 17
    sizes = [5, 70, 3, 114]
    offs, n, ld = _layout(sizes)
    assert ld == n
    pal = [F(5, 2), F(4, 3)]
    opal = [ofmt(f) for f in pal]
    fmt_idx = np.array([0, 1, 0, 1], np.uint8)
    G = _values(rng, W, ld, offs, "normal")
    G_t = torch.from_numpy(G).to(dev)
    offs_t = torch.from_numpy(offs).to(dev)
    idx_t = torch.from_numpy(fmt_idx).to(dev)
    mab = torch.zeros(len(sizes), dtype=torch.int32, device=dev)
    A.aps_layer_maxabs(G_t, n, offs_t, mab)
    o_mab = O.layer_maxabs(G, n, offs)
    o_se = O.layer_scales(o_mab, W, opal, fmt_idx)
    # every row's layers, one after another, for the oracle's packing
    offs_rows = np.append((offs[None, :-1] + n * np.arange(W, dtype=np.int64)[:, None]).ravel(), W * n)
    for mode, se in (("aps", o_se), ("raw", None)):
        se_t = None if se is None else torch.from_numpy(se).to(dev)
        Q_t = torch.zeros_like(G_t)
        codes_t = torch.zeros(W * n, dtype=torch.uint8, device=dev)
        A.aps_quantize(G_t, n, offs_t, se_t, pal, idx_t, Q=Q_t, codes=codes_t)
        torch.cuda.synchronize()
        assert same_maxabs(mab.cpu().numpy(), o_mab)
        o_Q = O.quantize(G, n, offs, se, opal, fmt_idx)
        Qg = Q_t.cpu().numpy()
        assert same_f32(Qg, o_Q), (mode, first_diff(Qg, o_Q))
        o_codes = O.pack_codes(o_Q.ravel(), offs_rows, opal, np.tile(fmt_idx, W))
        assert np.array_equal(codes_t.cpu().numpy(), o_codes), mode
        log(f"quantize W={W} mixed palette {mode}: values and codes match")


@pytest.mark.parametrize("n_total", [1, 2, 3, 4, 5, 7, 9])
def test_tiny_gradients(dev, n_total):
    """Gradients of a few elements, fewer than one thread's 4 or just past
    them: every call, in one layer and in two, in APS and RAW mode."""
    seed = zlib.crc32(f"tiny/{n_total}".encode())
    rng = np.random.default_rng(seed)
    for sizes in ([n_total], [n_total // 2, n_total - n_total // 2]):
        offs, n, ld = _layout(sizes)
        for f in (F(5, 2), F(3, 0), F(5, 10)):
            for W in (1, 3):
                G = _values(rng, W, ld, offs, "normal")
                tag = f"{f} sizes={sizes} W={W} seed={seed}"
                log("case", tag)
                run_case(dev, G, n, offs, [f], mode="aps", tag=tag + " aps")
                run_case(dev, G, n, offs, [f], mode="raw", tag=tag + " raw")


@pytest.mark.parametrize("f", [F(5, 2), F(3, 0), F(5, 10), F(8, 7, 130)], ids=str)
def test_quantize_in_place_and_dequantize_in_place(dev, f):
    """The header lets Q alias X (aps_quantize) and out alias Q
    (aps_dequantize): both in place, on the edge layout with specials, equal
    the oracle's out-of-place results."""
    seed = zlib.crc32(f"in-place/{f}".encode())
    rng = np.random.default_rng(seed)
    offs, n, ld = _layout(SIZES)
    opal = [ofmt(f)]
    for W in (1, 3):
        G = _values(rng, W, ld, offs, "special")
        se = rng.integers(-40, 40, offs.size - 1).astype(np.int32)
        X_t = torch.from_numpy(G).to(dev)
        offs_t = torch.from_numpy(offs).to(dev)
        se_t = torch.from_numpy(se).to(dev)
        A.aps_quantize(X_t, n, offs_t, se_t, [f], None, Q=X_t)
        torch.cuda.synchronize()
        o_Q = O.quantize(G, n, offs, se, opal)
        got = X_t.cpu().numpy()
        assert same_f32(got[:, :n], o_Q[:, :n]), f"{f} W={W} seed={seed} quantize in place"
        # the padding past n is left as it was
        assert same_f32(got[:, n:], G[:, n:]), f"{f} W={W} padding"
        row = X_t[0, :].contiguous()
        A.aps_dequantize(row, None, n, offs_t, se_t, [f], None, row)
        torch.cuda.synchronize()
        o_d = O.dequantize(o_Q[0, :n], None, n, offs, se, opal)
        assert same_f32(row.cpu().numpy()[:n], o_d), f"{f} W={W} seed={seed} dequantize in place"


def test_empty_gradient(dev):
    offs = np.zeros(4, np.int64)
    G = np.zeros((3, 4), np.float32)
    G_t = torch.from_numpy(G).to(dev)
    offs_t = torch.from_numpy(offs).to(dev)
    mab = torch.full((3,), 7, dtype=torch.int32, device=dev)
    A.aps_layer_maxabs(G_t, 0, offs_t, mab)
    assert mab.cpu().tolist() == [0, 0, 0]
    A.aps_sim_reduce(G_t, 0, offs_t, None, [F(5, 2)], None, 0, out=None)
    torch.cuda.synchronize()


# ------------------------------------------------ exhaustive small formats

SMALL = [F(5, 2), F(4, 3), F(3, 0), F(2, 0), F(2, 1), F(3, 2), F(6, 1), F(3, 4), F(4, 3, 5),
         F(4, 3, 140), F(3, 0, 145), F(2, 1, 147), F(5, 2, 140), F(8, 1, 140), F(3, 12)]


@pytest.mark.parametrize("f", SMALL, ids=str)
def test_every_code_and_midpoint(dev, f):
    vals = [float(v) for v in X.values(f.e, f.m, f.b)]
    ext = vals + [2.0 ** (f.emax + 1)]
    pts = list(vals)
    for lo, hi in zip(ext[:-1], ext[1:]):
        mid = np.float32((lo + hi) / 2)
        pts += [float(mid), float(np.nextafter(mid, np.float32(0))), float(np.nextafter(mid, np.float32(np.inf)))]
    pts = np.array(pts + [-p for p in pts] + [np.inf, -np.inf, np.nan], np.float32)
    n = pts.size
    ld = (n + 63) // 64 * 64
    G = np.full((1, ld), np.nan, np.float32)
    G[0, :n] = pts
    offs = np.array([0, n], np.int64)
    run_case(dev, G, n, offs, [f], mode="raw", tag=f"{f} all codes/midpoints")


@pytest.mark.parametrize("f", [F(5, 2), F(4, 3), F(3, 0), F(2, 1), F(3, 2), F(4, 3, 140), F(3, 0, 145),
                               F(5, 2, 140)], ids=str)
def test_every_code_pair_sum(dev, f):
    vals = [float(v) for v in X.values(f.e, f.m, f.b)]
    vals = np.array(vals + [-v for v in vals[1:]] + [np.inf, -np.inf], np.float32)
    a, b = np.meshgrid(vals, vals, indexing="ij")
    n = a.size
    ld = (n + 63) // 64 * 64
    G = np.zeros((2, ld), np.float32)
    G[0, :n] = a.ravel()
    G[1, :n] = b.ravel()
    offs = np.array([0, n], np.int64)
    G_t = torch.from_numpy(G).to(dev)
    offs_t = torch.from_numpy(offs).to(dev)
    out = torch.zeros(n, dtype=torch.float32, device=dev)
    flags = A.APS_INPUT_QUANTIZED | A.APS_OUTPUT_SCALED
    A.aps_sim_reduce(G_t, n, offs_t, None, [f], None, flags, out=out)
    o = O.sim_reduce(G, n, offs, None, ofmt(f), flags=O.INPUT_QUANTIZED | O.OUTPUT_SCALED)
    g = out.cpu().numpy()
    assert same_f32(g, o), first_diff(g, o)


# ----------------------------------------------------- paper-shaped sets

def _small_config(dev, name, palette):
    gs = WL.generate(name, palette, device="cpu")
    G = gs.G.numpy()
    pal = [A.Format(p.e, p.m, p.bias) for p in gs.palette]
    return G, gs, pal


@pytest.mark.parametrize("name,palette", [("mlp", "1-4-3"), ("resnet20", "1-5-2"), ("resnet20", "1-4-3"),
                                          ("resnet20", "1-3-0")])
def test_config_full_parity(dev, name, palette):
    G, gs, pal = _small_config(dev, name, palette)
    log("config", name, palette, G.shape)
    run_case(dev, G, gs.n, gs.offsets, pal, fmt_idx=gs.fmt_idx, mode="aps", tag=f"{name} {palette} aps")
    run_case(dev, G, gs.n, gs.offsets, pal, fmt_idx=gs.fmt_idx, mode="raw", tag=f"{name} {palette} raw")


def _sample_idx(rng, offs, n, per=20000):
    """Sorted unique sample of element indices: layer edges, chunk edges, random."""
    picks = [rng.integers(0, n, per)]
    for o in offs[1:-1]:
        picks.append(np.arange(max(0, o - 5), min(n, o + 5)))
    picks.append(np.arange(0, min(n, 2048)))
    picks.append(np.arange(max(0, n - 2048), n))
    picks.append((np.arange(0, n, 1024 * 997))[:200])
    idx = np.unique(np.concatenate(picks))
    return idx[(idx >= 0) & (idx < n)]


def _sampled_oracle(G_t, gs, pal, idx, o_se, fmt_idx, W):
    """Oracle on the sampled columns: same bytes, same per-layer exponents."""
    idx_t = torch.from_numpy(idx).to(G_t.device)
    Gs = G_t[:, idx_t].cpu().numpy()                       # [W][S]
    layer = np.searchsorted(gs.offsets, idx, side="right") - 1
    uniq, starts = np.unique(layer, return_index=True)
    sub_offs = np.append(starts, idx.size).astype(np.int64)
    se = None if o_se is None else o_se[uniq]
    fi = None if fmt_idx is None else fmt_idx[uniq]
    S = idx.size
    ldS = (S + 3) // 4 * 4
    Gp = np.zeros((W, ldS), np.float32)
    Gp[:, :S] = Gs
    return O.sim_reduce(Gp, S, sub_offs, se, [ofmt(f) for f in pal], fi)


def _oracle_maxabs_streamed(G_t, gs, rows=8):
    """Oracle max-abs of a large set, a few worker rows at a time."""
    W = G_t.shape[0]
    acc = np.zeros(gs.offsets.size - 1, np.uint32)
    for w0 in range(0, W, rows):
        part = G_t[w0:w0 + rows].cpu().numpy()
        m = O.layer_maxabs(part, gs.n, gs.offsets).view(np.uint32)
        acc = np.maximum(acc, m)
    return acc


@pytest.mark.parametrize("name,palette", [("resnet50_w8", "1-5-2"), ("resnet50_w256", "1-5-2"),
                                          ("resnet50_w256", "1-4-3"), ("bert_large", "hybrid")])
def test_config_large_parity(dev, name, palette):
    t0 = time.time()
    gs = WL.generate(name, palette, device=dev)
    G_t = gs.G
    W, n = gs.W, gs.n
    pal = [A.Format(p.e, p.m, p.bias) for p in gs.palette]
    opal = [ofmt(f) for f in pal]
    offs_t = torch.from_numpy(gs.offsets).to(dev)
    idx_t = None if gs.fmt_idx is None else torch.from_numpy(gs.fmt_idx).to(dev)
    log(name, palette, "generated", tuple(G_t.shape), f"{time.time() - t0:.1f}s")
    out, se_t, mab = A.aps_step(G_t, n, offs_t, pal, idx_t)
    torch.cuda.synchronize()
    log("gpu step done", f"{time.time() - t0:.1f}s")
    o_mab = _oracle_maxabs_streamed(G_t, gs)
    assert same_maxabs(mab.cpu().numpy(), o_mab), "maxabs"
    o_se = O.layer_scales(o_mab, W, opal, gs.fmt_idx)
    assert np.array_equal(se_t.cpu().numpy(), o_se), "scales"
    log("maxabs/scales match", f"{time.time() - t0:.1f}s")
    rng = np.random.default_rng(7)
    if name == "resnet50_w8":
        G = G_t.cpu().numpy()
        o_out = O.sim_reduce(G, n, gs.offsets, o_se, opal, gs.fmt_idx)
        g = out.cpu().numpy()
        assert same_f32(g, o_out), first_diff(g, o_out)
        assert np.all(np.isfinite(g))
        log("full reduce parity", f"{time.time() - t0:.1f}s")
    else:
        idx = _sample_idx(rng, gs.offsets, n)
        o_s = _sampled_oracle(G_t, gs, pal, idx, o_se, gs.fmt_idx, W)
        g = out[torch.from_numpy(idx).to(dev)].cpu().numpy()
        assert same_f32(g, o_s), first_diff(g, o_s)
        log("sampled reduce parity on", idx.size, f"{time.time() - t0:.1f}s")
    # APS mode never overflows on finite gradients
    assert bool(torch.isfinite(out).all())
    del G_t, gs
    torch.cuda.empty_cache()


def test_run_to_run_determinism(dev):
    gs = WL.generate("resnet20", "1-5-2", device=dev)
    offs_t = torch.from_numpy(gs.offsets).to(dev)
    pal = [A.Format(5, 2)]
    a, _, _ = A.aps_step(gs.G, gs.n, offs_t, pal)
    b, _, _ = A.aps_step(gs.G, gs.n, offs_t, pal)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


@pytest.mark.parametrize("f", [F(5, 2), F(4, 3), F(3, 0), F(2, 1), F(5, 10), F(8, 7), F(3, 4), F(4, 3, 5),
                               F(4, 3, 140), F(3, 2, 140), F(5, 10, 120), F(3, 0, 145)], ids=str)
def test_sim_reduce_codes_random_codes(dev, f):
    """Every code value (INF and NaN codes included) as input to the codes reduce."""
    rng = np.random.default_rng(40 + f.e * 3 + f.m)
    cls = _code_cls(f.bits)
    sizes = [0, 5, 4096, 31, 1, 8191, 3, 600]
    offs = np.zeros(len(sizes) + 1, np.int64)
    offs[1:] = np.cumsum(sizes)
    n = int(offs[-1])
    ld = (n + 63) // 64 * 64
    for W in (1, 2, 7, 16):
        codes = rng.integers(0, 1 << f.bits, (W, ld))
        if cls == 0:
            rows = np.zeros((W, ld // 2), np.uint8)
            rows[:] = (codes[:, 0::2] & 15) | ((codes[:, 1::2] & 15) << 4)
        elif cls == 1:
            rows = codes.astype(np.uint8)
        else:
            rows = codes.astype("<u2").view(np.uint8).reshape(W, -1)
        se = rng.integers(-20, 20, len(sizes)).astype(np.int32)
        c_t = torch.from_numpy(np.ascontiguousarray(rows).reshape(-1)).to(dev)
        offs_t = torch.from_numpy(offs).to(dev)
        se_t = torch.from_numpy(se).to(dev)
        out = torch.zeros(n, dtype=torch.float32, device=dev)
        A.aps_sim_reduce_codes(c_t, W, ld, n, offs_t, se_t, [f], None, 0, out=out)
        o = O.sim_reduce_codes(rows, W, ld, n, offs, se, ofmt(f))
        g = out.cpu().numpy()
        assert same_f32(g, o), (f, W, first_diff(g, o))



# ------------------------------------------- summation orders and Kahan

def _run_ex(dev, G, n, offs, pal, fmt_idx, se, k, acc, tag):
    W, ld = G.shape
    G_t = torch.from_numpy(G).to(dev)
    offs_t = torch.from_numpy(offs).to(dev)
    idx_t = None if fmt_idx is None else torch.from_numpy(fmt_idx).to(dev)
    se_t = None if se is None else torch.from_numpy(se).to(dev)
    out = torch.zeros(max(n, 1), dtype=torch.float32, device=dev)
    A.aps_sim_reduce_ex(G_t, n, offs_t, se_t, pal, idx_t, 0, group=k, accumulator=acc, out=out)
    o = O.sim_reduce_ex(G, n, offs, se, [ofmt(f) for f in pal], fmt_idx, group=k, accumulator=acc)
    g = out.cpu().numpy()[:n]
    assert same_f32(g, o), f"{tag} {first_diff(g, o)}"


@pytest.mark.parametrize("acc", [A.APS_ACC_SEQUENTIAL, A.APS_ACC_KAHAN])
@pytest.mark.parametrize("f", [F(5, 2), F(4, 3), F(3, 0), F(5, 10), F(8, 7), F(5, 12), F(8, 23), F(8, 7, 130),
                               F(5, 10, 120), F(3, 0, 145)], ids=str)
def test_ordered_reduce_edge_layouts(dev, f, acc):
    rng = np.random.default_rng(60 + f.e * 5 + f.m + 100 * acc)
    offs, n, ld = _layout(SIZES)
    for W, k in ((8, 1), (8, 2), (8, 8), (16, 4), (12, 4), (5, 1), (1, 1)):
        G = _values(rng, W, ld, offs, "special" if W % 2 else "normal")
        mab = O.layer_maxabs(G, n, offs)
        se = O.layer_scales(mab, W, ofmt(f))
        log("case", f, W, k, acc)
        _run_ex(dev, G, n, offs, [f], None, se, k, acc, f"{f} W={W} k={k} acc={acc}")


@pytest.mark.parametrize("acc", [A.APS_ACC_SEQUENTIAL, A.APS_ACC_KAHAN])
def test_ordered_reduce_mixed_palette(dev, acc):
    rng = np.random.default_rng(70 + acc)
    pal = [F(5, 2), F(4, 3), F(5, 10)]
    sizes = [int(v) for v in rng.choice([0, 1, 3, 17, 1000, 1023, 1024, 3000], 30)]
    offs, n, ld = _layout(sizes)
    fmt_idx = rng.integers(0, len(pal), len(sizes)).astype(np.uint8)
    G = _values(rng, 16, ld, offs, "normal")
    _run_ex(dev, G, n, offs, pal, fmt_idx, None, 2, acc, "mixed k=2")
    _run_ex(dev, G, n, offs, pal, fmt_idx, None, 1, acc, "mixed ring")


@pytest.mark.parametrize("k,acc", [(1, 0), (2, 0), (4, 1), (8, 1)])
def test_ordered_reduce_resnet50_w8_full(dev, k, acc):
    gs = WL.generate("resnet50_w8", "1-5-2", device=dev)
    G_t = gs.G
    offs_t = torch.from_numpy(gs.offsets).to(dev)
    pal = [F(5, 2)]
    _, se_t, _ = A.aps_step(G_t, gs.n, offs_t, pal)
    out = torch.empty(gs.n, dtype=torch.float32, device=dev)
    A.aps_sim_reduce_ex(G_t, gs.n, offs_t, se_t, pal, None, 0, group=k, accumulator=acc, out=out)
    G = G_t.cpu().numpy()
    o = O.sim_reduce_ex(G, gs.n, gs.offsets, se_t.cpu().numpy(), ofmt(pal[0]), group=k, accumulator=acc)
    g = out.cpu().numpy()
    assert same_f32(g, o), first_diff(g, o)
    assert np.all(np.isfinite(g))


def test_ordered_reduce_w256_groups(dev):
    """W = 256 with the paper's group sizes on a 1.1 M-element ResNet-like slice."""
    rng = np.random.default_rng(80)
    sizes = [9408, 64, 64, 4096, 64, 64, 36864, 64, 64, 16384, 256, 256, 16384, 256, 256, 1000000, 1000]
    offs, n, ld = _layout(sizes)
    W = 256
    G = np.zeros((W, ld), np.float32)
    for i, sz in enumerate(sizes):
        a, b = offs[i], offs[i + 1]
        G[:, a:b] = (rng.standard_normal((W, sz)) * 10.0 ** rng.uniform(-7, -1)).astype(np.float32)
    mab = O.layer_maxabs(G, n, offs)
    se = O.layer_scales(mab, W, O.Format(5, 2))
    for k in (1, 16, 64):
        log("W=256 k", k)
        _run_ex(dev, G, n, offs, [F(5, 2)], None, se, k, A.APS_ACC_SEQUENTIAL, f"W=256 k={k}")


# ------------------------------- low-precision-accumulator GEMM (Sec. 5, CPD)

# (input format, accumulator format): every accumulator variant of the kernel
GEMM_PAIRS = [
    (F(5, 2), F(5, 2)),     # TOP class, fp32 adds
    (F(4, 3), F(4, 3)),     # LOW class
    (F(4, 3), F(5, 2)),
    (F(5, 10), F(5, 10)),   # fp16
    (F(8, 7), F(8, 7)),     # bf16: INT class, products below fp32's normal range
    (F(5, 10), F(8, 23)),   # fp32 accumulator
    (F(5, 2), F(6, 12)),    # TOP class, fp64 adds
    (F(3, 2), F(3, 12)),    # LOW class, fp64 adds
    (F(5, 10), F(8, 15)),   # INT class, fp64 adds
    (F(4, 3), F(5, 0)),     # m = 0, TOP class
    (F(2, 1), F(2, 0)),     # m = 0, LOW class: the 3-bit accumulator
    (F(8, 3), F(8, 0)),     # m = 0, INT class
    (F(5, 2), F(5, 10)),    # the accumulator is IEEE half: the hardware's half-precision arithmetic
    (F(5, 2, 16), F(5, 10)),  # the same from inputs of another bias
    (F(4, 2), F(5, 9)),     # products fit the accumulator's significand: TOP class (rounded on its grid)
    (F(4, 1), F(4, 6)),     # products fit: LOW class (rounded on its grid)
    (F(2, 1), F(4, 6)),     # products fit and never reach the subnormal range: LOW class, no rounding
    (F(3, 1), F(5, 7)),     # the same, TOP class
    (F(5, 2), F(8, 7)),     # the same into bfloat16: the adds rounded by the hardware's conversion
    (F(7, 1), F(8, 7)),     # bfloat16 again, with products overflowing and sums below 2^-126
    (F(4, 3), F(8, 7)),     # bfloat16 from LOW-class inputs
    (F(5, 0), F(8, 7)),     # bfloat16 from inputs with no mantissa bits
    (F(5, 2), F(8, 10)),    # exact products, INT class, not bfloat16
    (F(5, 2, 14), F(5, 10, 13)),  # 1-5-10 with another bias: not half, rounded on its grid
    (F(7, 1), F(7, 3)),     # products fit, but the accumulator spans 129 binades: the compare-and-select rounding
    (F(8, 3), F(5, 10)),    # bf16-range inputs cannot be pre-scaled: one ldexp per product, TOP
    (F(8, 2), F(4, 3)),     # the same, LOW class
]
GEMM_SHAPES = [(1, 1, 1), (70, 130, 37), (64, 64, 16), (5, 200, 0), (128, 96, 300), (3, 65, 17)]


def _gemm_inputs(rng, M, N, K, fin, specials=True):
    lo, hi = O.emin(ofmt(fin)) - fin.m - 1, max(O.emax(ofmt(fin)) // 2, 1)
    Am = (rng.standard_normal((M, K)) * 2.0 ** rng.uniform(lo, hi, (M, K))).astype(np.float32)
    Bm = (rng.standard_normal((K, N)) * 2.0 ** rng.uniform(lo, hi, (K, N))).astype(np.float32)
    if specials and M * K > 8 and K * N > 8:
        for arr in (Am, Bm):
            flat = arr.reshape(-1)
            idx = rng.choice(flat.size, 6, replace=False)
            flat[idx] = [0.0, -0.0, np.inf, -np.inf, np.nan, 3.0e38]
    return Am, Bm


@pytest.mark.parametrize("acc", [A.APS_ACC_SEQUENTIAL, A.APS_ACC_KAHAN])
@pytest.mark.parametrize("fin,facc", GEMM_PAIRS, ids=lambda f: str(f))
def test_lp_gemm_parity(dev, fin, facc, acc):
    rng = np.random.default_rng(900 + 7 * fin.e + facc.m + 31 * acc)
    for M, N, K in GEMM_SHAPES:
        for specials in (False, True):
            Am, Bm = _gemm_inputs(rng, M, N, K, fin, specials)
            log(f"lp_gemm {fin}->{facc} acc={acc} M={M} N={N} K={K} specials={specials}")
            got = A.aps_lp_gemm(torch.from_numpy(Am).to(dev), torch.from_numpy(Bm).to(dev), fin, facc, acc)
            torch.cuda.synchronize()
            ref = O.lp_gemm(Am, Bm, ofmt(fin), ofmt(facc), acc)
            g = got.cpu().numpy()
            assert same_f32(g, ref), (fin, facc, acc, M, N, K, specials, first_diff(g, ref))


def _grid_edge_inputs(rng, M, K, N):
    # 1-5-2 values whose products land at the edges of 1-5-10: its subnormal
    # range (step 2^-24, products on and between the steps, halfway ties
    # included), its smallest normal 2^-14, and its overflow at 2^16
    sig = np.array([1.0, 1.25, 1.5, 1.75])

    def vals(shape, lo, hi):
        e = rng.integers(lo, hi + 1, shape)
        return (rng.choice([-1.0, 1.0], shape) * rng.choice(sig, shape) * np.exp2(e)).astype(np.float32)

    Am = vals((M, K), -14, 8)
    Bm = vals((K, N), -14, 8)
    # rows of A small and columns of B small: products around 2^-28 .. 2^-10;
    # the other rows and columns large: products around 2^12 .. 2^17
    Am[: M // 2] = vals((M // 2, K), -14, -5)
    Bm[:, : N // 2] = vals((K, N // 2), -14, -5)
    Am[M // 2:] = vals((M - M // 2, K), 5, 8)
    Bm[:, N // 2:] = vals((K, N - N // 2), 5, 8)
    return Am, Bm


@pytest.mark.parametrize("shift", [0, 1], ids=["half", "bias-shifted"])
@pytest.mark.parametrize("acc", [A.APS_ACC_SEQUENTIAL, A.APS_ACC_KAHAN])
def test_lp_gemm_product_grid_edges(dev, acc, shift):
    """1-5-2 inputs, a 1-5-10 accumulator: products rounded on the
    accumulator's subnormal grid (ties to even), at its smallest normal, and
    at its overflow with a partial sum of the other sign already there.  With
    shift 1 every input is doubled and both biases lowered by one and two:
    the same chains at 4 times the scale, in formats that are not IEEE half
    (the kernel rounds them on the grid instead of in half precision)."""
    fin, facc = F(5, 2, 15 - shift), F(5, 10, 15 - 2 * shift)
    # hand-made chains of two products (row i of A with column i of B)
    cases = [
        ((1.75 * 2 ** 7, 2.0 ** 8), (-(2.0 ** 8), 2.0 ** 8)),         # -57344, then 2^16 overflows: INF
        ((1.75 * 2 ** 7, 1.75 * 2 ** 7), (-(2.0 ** 8), 2.0 ** 8)),    # -57344 + 57344 = 0
        ((1.25 * 2 ** -12, 1.5 * 2 ** -12), (2.0 ** -11, 2.0 ** -12)),  # 2.5 and 1.5 steps: ties to 2 and 2
        ((2.0 ** -12, 1.5 * 2 ** -13), (2.0 ** -13, 2.0 ** -12)),     # 0.5 step (to 0), 0.75 step (to 1)
        ((1.75 * 2 ** -8, 2.0 ** -7), (1.75 * 2 ** -8, 2.0 ** -7)),   # 784 steps, then 2^-14 itself
        ((-1.25 * 2 ** -12, 2.0 ** -12), (2.0 ** -11, -(2.0 ** -13))),  # -2.5 steps (to -2), -0.5 (to -0)
        ((2.0 ** 8, 1.5 * 2 ** -12), (-(2.0 ** 8), 2.0 ** -12)),      # overflow to -INF first, then a tiny one
    ]
    n = len(cases)
    Am = np.zeros((n, 2), np.float32)
    Bm = np.zeros((2, n), np.float32)
    for i, (a, b) in enumerate(cases):
        Am[i] = a
        Bm[:, i] = b
    rng = np.random.default_rng(1210 + acc)
    for tag, (Ax, Bx) in (("hand-made", (Am, Bm)), ("random K=64", _grid_edge_inputs(rng, 96, 64, 80)),
                          ("random K=300", _grid_edge_inputs(rng, 70, 300, 70))):
        log(f"lp_gemm grid edges {tag} acc={acc}")
        Ax, Bx = Ax * np.float32(2 ** shift), Bx * np.float32(2 ** shift)
        got = A.aps_lp_gemm(torch.from_numpy(Ax).to(dev), torch.from_numpy(Bx).to(dev), fin, facc, acc)
        torch.cuda.synchronize()
        ref = O.lp_gemm(Ax, Bx, ofmt(fin), ofmt(facc), acc)
        g = got.cpu().numpy()
        assert same_f32(g, ref), (tag, first_diff(g, ref))
        if tag == "hand-made":
            d = np.diag(ref) / 4.0 ** shift
            assert d[0] == np.inf and d[1] == 0.0 and d[6] == -np.inf
            assert d[2] == 4 * 2.0 ** -24 and d[3] == 2.0 ** -24 and d[4] == 784 * 2.0 ** -24 + 2.0 ** -14
            assert d[5] == -2 * 2.0 ** -24


@pytest.mark.parametrize("acc", [A.APS_ACC_SEQUENTIAL, A.APS_ACC_KAHAN])
def test_lp_gemm_bfloat16_edges(dev, acc):
    """1-7-1 inputs into a bfloat16 accumulator (every product exact, the
    adds rounded by the hardware's conversion to bfloat16): halfway sums
    (ties to even), overflow of a sum to INF, cancellation, and products from
    the inputs' smallest subnormal to beyond bfloat16's range."""
    fin, facc = F(7, 1), F(8, 7)
    big = 1.5 * 2.0 ** 63
    cases = [  # (row of A, column of B): K = 3
        ((1.0, 2.0 ** -4, 0.0), (1.0, 2.0 ** -4, 0.0)),                  # 1 + 2^-8: a tie, to 1
        ((1.0, 2.0 ** -4, 2.0 ** -4), (1.0, 2.0 ** -3, 2.0 ** -4)),      # 1 + 2^-7, then + 2^-8: a tie, to 1 + 2^-6
        ((big, big, 0.0), (big, big, 0.0)),                              # 2.25 * 2^126 twice: INF (Kahan: NaN next)
        ((big, big, 1.0), (big, -big, 1.0)),                             # cancels to 0, then 1
        ((big, 2.0 ** 63, big), (2.0 ** 63, 2.0 ** 63, big)),            # 1.5 * 2^126 + 2^126 + 2.25 * 2^126: INF
        ((2.0 ** -63, 1.0, -1.0), (2.0 ** -63, 2.0 ** -40, 2.0 ** -40)),  # 2^-126 swamped by 2^-40, then cancelled
    ]
    n = len(cases)
    Am = np.zeros((n, 3), np.float32)
    Bm = np.zeros((3, n), np.float32)
    for i, (a, b) in enumerate(cases):
        Am[i] = a
        Bm[:, i] = b
    rng = np.random.default_rng(1230 + acc)
    for tag, (Ax, Bx) in (("hand-made", (Am, Bm)), ("random", _gemm_inputs(rng, 70, 80, 300, fin))):
        log(f"lp_gemm bfloat16 edges {tag} acc={acc}")
        got = A.aps_lp_gemm(torch.from_numpy(Ax).to(dev), torch.from_numpy(Bx).to(dev), fin, facc, acc)
        torch.cuda.synchronize()
        ref = O.lp_gemm(Ax, Bx, ofmt(fin), ofmt(facc), acc)
        g = got.cpu().numpy()
        assert same_f32(g, ref), (tag, first_diff(g, ref))
        if tag == "hand-made":
            d = np.diag(ref)
            assert d[0] == 1.0 and d[1] == 1.0 + 2.0 ** -6 and d[3] == 1.0 and d[4] == np.inf and d[5] == 0.0
            # an INF partial sum with zero added: plain stays INF; Kahan's compensation is INF by then,
            # so the next add is INF - INF
            assert d[2] == np.inf if acc == A.APS_ACC_SEQUENTIAL else np.isnan(d[2])


def _cast_boundary_values():
    # fp32 values at every rounding position of 1-5-2: both signs, every
    # exponent field (zeros, subnormals, INF and NaN among them), the top six
    # mantissa bits in all combinations (round bit and the bits above it for
    # the normal and subnormal grids alike) and four patterns of the bits
    # below (none set, the lowest, the highest, all)
    sign = np.arange(2, dtype=np.uint32)[:, None, None, None] << 31
    expo = np.arange(256, dtype=np.uint32)[None, :, None, None] << 23
    top = np.arange(64, dtype=np.uint32)[None, None, :, None] << 17
    low = np.array([0, 1, 0x10000, 0x1FFFF], dtype=np.uint32)[None, None, None, :]
    return (sign | expo | top | low).reshape(-1).view(np.float32)


@pytest.mark.parametrize("facc", [F(5, 10), F(5, 7), F(8, 7)], ids=["half", "grid", "exact-bf16"])
@pytest.mark.parametrize("fin", [F(5, 2), F(4, 3)], ids=str)
def test_lp_gemm_input_cast_rounding_cases(dev, fin, facc):
    """1-5-2 and 1-4-3 inputs (the formats the GEMM casts by the hardware's
    8-bit float conversions) at every rounding case of their cast (ties,
    sticky bits, the subnormal grid, overflow to INF, NaN, signed zeros),
    each times 1.0 with zeros in the other k slots, in whole tiles so that
    the half kernel casts its staged values two at a time."""
    x = _cast_boundary_values()
    M, K, N = x.size, 16, 64
    Am = np.zeros((M, K), np.float32)
    Am[:, 0] = x
    Bm = np.zeros((K, N), np.float32)
    Bm[0, :] = 1.0
    log(f"lp_gemm input cast cases {fin}->{facc} M={M}")
    got = A.aps_lp_gemm(torch.from_numpy(Am).to(dev), torch.from_numpy(Bm).to(dev), fin, facc).cpu().numpy()
    ref = O.lp_gemm(Am, np.ascontiguousarray(Bm[:, :1]), ofmt(fin), ofmt(facc))
    assert same_f32(got[:, :1], ref), first_diff(got[:, :1], ref)
    assert same_f32(got, np.repeat(got[:, :1], N, axis=1))


@pytest.mark.parametrize("fin,facc", [(F(5, 2), F(5, 10)), (F(4, 3), F(5, 2))], ids=["half", "emulated"])
@pytest.mark.parametrize("M,N", [(1 << 22, 3), (2, 1 << 22)])
def test_lp_gemm_largest_dimensions(dev, M, N, fin, facc):
    """M or N at APS_MAX_GEMM_DIM = 2^22: 65536 tiles along one dimension,
    in both GEMM kernels (half-precision accumulator, and the emulated one)."""
    rng = np.random.default_rng(977 + M % 7)
    Am, Bm = _gemm_inputs(rng, M, N, 2, fin)
    got = A.aps_lp_gemm(torch.from_numpy(Am).to(dev), torch.from_numpy(Bm).to(dev), fin, facc)
    torch.cuda.synchronize()
    ref = O.lp_gemm(Am, Bm, ofmt(fin), ofmt(facc))
    g = got.cpu().numpy()
    assert same_f32(g, ref), first_diff(g, ref)


@pytest.mark.parametrize("fin,facc", [(F(5, 2), F(5, 10)), (F(4, 3), F(5, 2))], ids=["half", "emulated"])
def test_lp_gemm_strided_views(dev, fin, facc):
    # row strides from the tensors (leading dimensions larger than the width)
    rng = np.random.default_rng(950)
    Abig = rng.standard_normal((40, 100)).astype(np.float32)
    Bbig = rng.standard_normal((77, 90)).astype(np.float32)
    At = torch.from_numpy(Abig).to(dev)[:, 3:80]
    Bt = torch.from_numpy(Bbig).to(dev)[:, 5:70]
    C = torch.full((40, 80), 7.0, device=dev)
    A.aps_lp_gemm(At, Bt, fin, facc, C=C[:, :65])
    torch.cuda.synchronize()
    ref = O.lp_gemm(Abig[:, 3:80], Bbig[:, 5:70], ofmt(fin), ofmt(facc))
    c = C.cpu().numpy()
    assert same_f32(c[:, :65], ref)
    assert (c[:, 65:] == 7.0).all()  # nothing written past N


@pytest.mark.parametrize("facc", [F(5, 10), F(5, 7), F(8, 7)], ids=["half", "grid", "exact-bf16"])
@pytest.mark.parametrize("acc", [A.APS_ACC_SEQUENTIAL, A.APS_ACC_KAHAN])
def test_lp_gemm_bert_ffn_sampled(dev, acc, facc):
    # BERT-large's first FFN product at 8 sequences of 512 tokens:
    # [4096 tokens x 1024] x [1024 x 4096], 1-5-2 inputs, the accumulators the
    # benchmark times (IEEE half; 1-5-7, products rounded on its grid;
    # bfloat16, exact products); sampled rows and columns against the oracle
    rng = np.random.default_rng(960 + acc)
    M, K, N = 4096, 1024, 4096
    fin = F(5, 2)
    Am = rng.standard_normal((M, K)).astype(np.float32)
    Bm = (rng.standard_normal((K, N)) * 0.02).astype(np.float32)
    log(f"lp_gemm BERT FFN M={M} K={K} N={N} acc={acc} into {facc}")
    got = A.aps_lp_gemm(torch.from_numpy(Am).to(dev), torch.from_numpy(Bm).to(dev), fin, facc, acc)
    torch.cuda.synchronize()
    g = got.cpu().numpy()
    rows = np.sort(rng.choice(M, 6, replace=False))
    cols = np.sort(rng.choice(N, 6, replace=False))
    ref_r = O.lp_gemm(Am[rows], Bm, ofmt(fin), ofmt(facc), acc)
    assert same_f32(g[rows], ref_r), first_diff(g[rows], ref_r)
    ref_c = O.lp_gemm(Am, np.ascontiguousarray(Bm[:, cols]), ofmt(fin), ofmt(facc), acc)
    assert same_f32(g[:, cols], ref_c), first_diff(g[:, cols], ref_c)


@pytest.mark.parametrize("f", [F(3, 0), F(5, 0), F(8, 0), F(5, 2), F(5, 10)], ids=str)
def test_kahan_compensation_nan_does_not_reach_the_sum(dev, f):
    # s = INF, then x = 1: t = INF, but the compensation R(R(t - s) - y) is
    # NaN; the sum itself stays INF (m = 0 formats included)
    G = np.array([[np.inf] * 8, [1.0] * 8], np.float32)
    offs = np.array([0, 8], np.int64)
    ref = O.sim_reduce_ex(G, 8, offs, None, ofmt(f), accumulator=O.ACC_KAHAN)
    assert np.isinf(ref).all()
    out = torch.empty(8, device=dev)
    A.aps_sim_reduce_ex(torch.from_numpy(G).to(dev), 8, torch.from_numpy(offs).to(dev), None, [f], None, 0,
                        accumulator=A.APS_ACC_KAHAN, out=out)
    torch.cuda.synchronize()
    assert same_f32(out.cpu().numpy(), ref)
    # the same chain as a dot product: products INF * 1 and 1 * 1
    Am = np.array([[np.inf, 1.0]], np.float32)
    Bm = np.array([[1.0], [1.0]], np.float32)
    fin = F(5, 2) if f.e < 8 else F(8, 3)
    refg = O.lp_gemm(Am, Bm, ofmt(fin), ofmt(f), O.ACC_KAHAN)
    got = A.aps_lp_gemm(torch.from_numpy(Am).to(dev), torch.from_numpy(Bm).to(dev), fin, f, A.APS_ACC_KAHAN)
    torch.cuda.synchronize()
    assert np.isinf(refg).all() and same_f32(got.cpu().numpy(), refg)
