"""Every element of the HBM-sized paper-shaped sets against the oracle.

The ResNet-50 sets (W = 8 and W = 256) and the BERT-large hybrid set are too
large for the oracle to take in one call of a few seconds, but not for the
oracle itself: the set is copied to host memory once, the oracle takes the
layer maxima on blocks of worker rows in parallel threads (the maximum of
bit patterns does not depend on how the rows are grouped), and the rounded
W-worker sum (Algorithm 1 with the low-precision accumulator of Sec. 5) on
successive column slices of all W rows, each slice with the full layers'
exponents.  Every output element of the HIP path is then compared with the
oracle's: fp32 bit patterns, NaN as a class.

Per (set, format, mode):
  * APS mode: maxima and scale exponents, then the sum of the two-pass
    calls (aps_layer_maxabs, aps_layer_scales, aps_sim_reduce), of aps_sync
    on its default route, and of aps_sync forced onto the one-pass and the
    guessed-scale routes;
  * RAW mode ("without APS", every exponent 0): aps_sim_reduce with no
    exponents.
The smaller sets (MLP, ResNet-20) are compared in full in test_gpu_parity.py
and test_gpu_sync.py."""
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle as O
from paper_1911_08907_amd import aps as A
from paper_1911_08907_amd import workloads as WL
from tests._util import first_diff, log, ofmt, same_f32, same_maxabs
from tests.oracle_stream import THREADS, oracle_maxabs, oracle_sum_sliced
from tests.test_gpu_parity import _sample_idx, _sampled_oracle

pytestmark = pytest.mark.gpu

@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    A.lib()  # the HIP library must be there: no fallback
    return torch.device("cuda:0")


class _Held:
    """One generated set at a time (device tensor and its host copy), shared
    by the tests of the same set and freed before the next set is drawn."""

    key = None
    gs = None
    host = None


@pytest.fixture(scope="module")
def held():
    yield _Held
    _release()


def _release():
    _Held.key = _Held.gs = _Held.host = None
    torch.cuda.empty_cache()


def _get(dev, name):
    if _Held.key != name:
        _release()
        t0 = time.time()
        gs = WL.generate(name, None, device=dev)
        torch.cuda.synchronize()
        host = gs.G.cpu().numpy()
        _Held.key, _Held.gs, _Held.host = name, gs, host
        log(name, "drawn and copied to the host", tuple(host.shape), f"{time.time() - t0:.1f}s")
    return _Held.gs, _Held.host


def _same_on_device(got, ref_t):
    """Bitwise equality of two fp32 device vectors, NaN as a class."""
    a, b = got.view(torch.int32), ref_t.view(torch.int32)
    both_nan = torch.isnan(got) & torch.isnan(ref_t)
    return bool(((a == b) | both_nan).all())


def _check(tag, got, o_out, ref_t):
    if not _same_on_device(got, ref_t):
        g = got.cpu().numpy()
        pytest.fail(f"{tag}: sum differs from the oracle {first_diff(g, o_out)}")
    log(f"  {tag}: all {o_out.size} elements equal the oracle's")


CASES = [("resnet50_w8", "1-5-2", "raw"),
         ("resnet50_w256", "1-5-2", "aps"), ("resnet50_w256", "1-5-2", "raw"),
         ("resnet50_w256", "1-4-3", "aps"), ("resnet50_w256", "1-4-3", "raw"),
         ("bert_large", "hybrid", "aps"), ("bert_large", "hybrid", "raw")]


@pytest.mark.parametrize("name,palette,mode", CASES, ids=[f"{a}-{b}-{c}" for a, b, c in CASES])
def test_every_element_against_the_oracle(dev, held, name, palette, mode):
    t0 = time.time()
    gs, host = _get(dev, name)
    G_t, W, n = gs.G, gs.W, gs.n
    cfg_pal = WL.CONFIGS[name].palettes[palette]
    pal = [A.Format(p.e, p.m, p.bias) for p in cfg_pal]
    opal = [ofmt(f) for f in pal]
    offs, fmt_idx = gs.offsets, gs.fmt_idx
    offs_t = torch.from_numpy(offs).to(dev)
    idx_t = None if fmt_idx is None else torch.from_numpy(fmt_idx).to(dev)
    tag = f"{name} {palette} {mode} W={W} n={n}"
    log(tag)

    if mode == "raw":
        out = torch.empty(n, dtype=torch.float32, device=dev)
        A.aps_sim_reduce(G_t, n, offs_t, None, pal, idx_t, 0, out=out)
        torch.cuda.synchronize()
        o_out = oracle_sum_sliced(host, n, offs, None, opal, fmt_idx, tag)
        ref_t = torch.from_numpy(o_out).to(dev)
        _check(f"{tag} aps_sim_reduce", out, o_out, ref_t)
        return

    o_mab = oracle_maxabs(host, n, offs)
    o_se = O.layer_scales(o_mab, W, opal, fmt_idx)
    log(f"  {tag}: oracle maxima and exponents {time.time() - t0:.1f}s")
    two, se, mab = A.aps_step(G_t, n, offs_t, pal, idx_t)
    results = {"two-pass calls": two}
    for route, flag in (("aps_sync default route", 0), ("aps_sync one pass", A.APS_SYNC_ONE_PASS),
                        ("aps_sync guessed scales", A.APS_SYNC_GUESS)):
        o, s2, m2, _ = A.aps_sync(G_t, n, offs_t, pal, idx_t, A.APS_SYNC_PASS1 | A.APS_SYNC_PASS2 | flag)
        torch.cuda.synchronize()
        assert same_maxabs(m2.cpu().numpy(), o_mab), f"{tag} {route}: maxima"
        assert np.array_equal(s2.cpu().numpy(), o_se), f"{tag} {route}: scale exponents"
        results[route] = o
    torch.cuda.synchronize()
    assert same_maxabs(mab.cpu().numpy(), o_mab), f"{tag}: maxima"
    assert np.array_equal(se.cpu().numpy(), o_se), f"{tag}: scale exponents"
    o_out = oracle_sum_sliced(host, n, offs, o_se, opal, fmt_idx, tag)
    assert np.all(np.isfinite(o_out)), "APS mode never overflows on finite gradients"
    ref_t = torch.from_numpy(o_out).to(dev)
    for route, got in results.items():
        _check(f"{tag} {route}", got, o_out, ref_t)
    log(f"  {tag}: done in {time.time() - t0:.1f}s")


def _boundary_rows(W, ld, row_bytes):
    """Rows around every place where a row's first element index or byte
    offset (fp32 values or codes) passes a multiple of 2^31, plus the first
    and last two rows; every row when there are few."""
    if W <= 16:
        return list(range(W))
    rows = {0, 1, W - 2, W - 1}
    for per_row in (ld, 4 * ld, row_bytes):
        k = 1
        while (k << 31) < W * per_row:
            r = (k << 31) // per_row
            rows.update(x for x in (r - 1, r, r + 1) if 0 <= x < W)
            k += 1
    return sorted(rows)


QCASES = [("resnet50_w8", "1-5-2"), ("resnet50_w256", "1-5-2"), ("resnet50_w256", "1-4-3"),
          ("bert_large", "hybrid")]


@pytest.mark.parametrize("name,palette", QCASES, ids=[f"{a}-{b}" for a, b in QCASES])
def test_quantize_codes_and_dequantize_full_rows(dev, held, name, palette):
    """aps_quantize (values and codes) on the whole set with the oracle's
    exponents, every element of every row at W = 8 and of the rows around
    each 2^31 boundary of the element index and of the value and code byte
    offsets at W = 256 (a 6.5 GB code array, 26 GB of values); the codes
    of two rows through aps_dequantize; all W rows of codes through
    aps_sim_reduce_codes, against the oracle's sum on sampled columns that
    include every layer edge.  A palette with mixed code widths writes no
    codes, so BERT-large checks the values only."""
    t0 = time.time()
    gs, host = _get(dev, name)
    G_t, W, n, ld = gs.G, gs.W, gs.n, gs.G.stride(0)
    cfg_pal = WL.CONFIGS[name].palettes[palette]
    pal = [A.Format(p.e, p.m, p.bias) for p in cfg_pal]
    opal = [ofmt(f) for f in pal]
    offs, fmt_idx = gs.offsets, gs.fmt_idx
    offs_t = torch.from_numpy(offs).to(dev)
    idx_t = None if fmt_idx is None else torch.from_numpy(fmt_idx).to(dev)
    bits = {f.bits for f in pal}
    codes = len({A.code_bytes(8, b) for b in bits}) == 1
    tag = f"{name} {palette} W={W} n={n}"
    o_se = O.layer_scales(oracle_maxabs(host, n, offs), W, opal, fmt_idx)
    se_t = torch.from_numpy(o_se).to(dev)
    rb = A.code_bytes(ld, max(bits))
    cb = A.code_bytes(n, max(bits))
    Q_t = torch.empty_like(G_t)
    codes_t = torch.zeros(W * rb, dtype=torch.uint8, device=dev) if codes else None
    A.aps_quantize(G_t, n, offs_t, se_t, pal, idx_t, Q=Q_t, codes=codes_t)
    torch.cuda.synchronize()
    rows = _boundary_rows(W, ld, rb if codes else 4 * ld)
    log(f"  {tag}: quantized; checking rows {rows} ({time.time() - t0:.1f}s)")
    for r0 in range(0, len(rows), 8):
        blk = rows[r0:r0 + 8]
        o_Q = O.quantize(np.ascontiguousarray(host[blk]), n, offs, o_se, opal, fmt_idx)
        g_Q = Q_t[torch.tensor(blk, device=dev), :n].cpu().numpy()
        assert same_f32(g_Q, o_Q[:, :n]), f"{tag} quantize rows {blk}: {first_diff(g_Q, o_Q[:, :n])}"
        if codes:
            def pack(i):
                return O.pack_codes(o_Q[i, :n], offs, opal, fmt_idx)
            with ThreadPoolExecutor(THREADS) as ex:
                o_codes = list(ex.map(pack, range(len(blk))))
            for i, w in enumerate(blk):
                g_c = codes_t[w * rb:w * rb + cb].cpu().numpy()
                assert np.array_equal(g_c, o_codes[i]), f"{tag} codes of row {w}"
            if r0 == 0:
                # two rows' codes decoded back: aps_dequantize against the oracle's
                for i in (0, len(blk) - 1):
                    w = blk[i]
                    out_t = torch.empty(n, dtype=torch.float32, device=dev)
                    A.aps_dequantize(None, codes_t[w * rb:(w + 1) * rb], n, offs_t, se_t, pal, idx_t, out_t)
                    o_d = O.dequantize(None, o_codes[i], n, offs, o_se, opal, fmt_idx)
                    assert same_f32(out_t.cpu().numpy(), o_d), f"{tag} dequantize row {w}"
        del o_Q, g_Q
    log(f"  {tag}: {len(rows)} rows of values" + (" and codes" if codes else "") +
        f" equal the oracle's ({time.time() - t0:.1f}s)")
    if codes and rb % 16 == 0:
        out_t = torch.empty(n, dtype=torch.float32, device=dev)
        A.aps_sim_reduce_codes(codes_t, W, ld, n, offs_t, se_t, pal, idx_t, 0, out=out_t)
        torch.cuda.synchronize()
        idx = _sample_idx(np.random.default_rng(11), offs, n)
        o_s = _sampled_oracle(G_t, gs, pal, idx, o_se, fmt_idx, W)
        g_s = out_t[torch.from_numpy(idx).to(dev)].cpu().numpy()
        assert same_f32(g_s, o_s), f"{tag} sim_reduce_codes {first_diff(g_s, o_s)}"
        log(f"  {tag}: sim_reduce_codes over all {W} rows equals the oracle on {idx.size} columns")
    del Q_t, codes_t
    torch.cuda.empty_cache()
    log(f"  {tag}: done in {time.time() - t0:.1f}s")
