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

import numpy as np
import pytest
import torch

import oracle as O
from paper_1911_08907_amd import aps as A
from paper_1911_08907_amd import workloads as WL
from tests._util import first_diff, log, ofmt, same_maxabs
from tests.oracle_stream import oracle_maxabs, oracle_sum_sliced

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

