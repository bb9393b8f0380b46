"""aps_sync_noalloc against aps_sync, through the C ABI.

aps_sync_noalloc is aps_sync with the library's static per-GPU workspace in
place of a caller's.  Its maxima, scale exponents and sums must equal, bit
for bit, what aps_sync returns on the same inputs with a workspace of its
own, on every route, with the passes issued together and separately.  The
array keeps the last call's contents, so each case makes two calls in a row,
the second on a smaller set, and a third call repeats the first set after a
call that fills the array with another set's bookkeeping.  The small set is
also checked against the oracle."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_1911_08907_amd import aps as A
from paper_1911_08907_amd import workloads as WL
from tests._util import first_diff, log, ofmt, same_f32, same_maxabs

pytestmark = pytest.mark.gpu

BOTH = A.APS_SYNC_PASS1 | A.APS_SYNC_PASS2
ROUTES = {"default": 0, "one pass": A.APS_SYNC_ONE_PASS, "guessed scales": A.APS_SYNC_GUESS,
          "two passes": A.APS_SYNC_TWO_PASS}


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    A.lib()  # the HIP library must be there: no fallback
    return torch.device("cuda:0")


class _Set:
    def __init__(self, name, palette, dev):
        gs = WL.generate(name, palette, device=dev)
        self.name, self.gs, self.G = f"{name} {palette}", gs, gs.G
        self.n, self.W, self.L = gs.n, gs.W, len(gs.sizes)
        self.pal = [A.Format(p.e, p.m, p.bias) for p in gs.palette]
        self.offs = torch.from_numpy(gs.offsets).to(dev)
        self.idx = None if gs.fmt_idx is None else torch.from_numpy(gs.fmt_idx).to(dev)


def _with_workspace(s, route):
    out, se, mab, _ = A.aps_sync(s.G, s.n, s.offs, s.pal, s.idx, BOTH | route)
    return out, se, mab


def _noalloc(s, route, split):
    dev = s.G.device
    mab = torch.full((s.L,), -1, dtype=torch.int32, device=dev)
    se = torch.full((s.L,), -7, dtype=torch.int32, device=dev)
    out = torch.full((s.n,), float("nan"), dtype=torch.float32, device=dev)
    if split:
        A.aps_sync_noalloc(s.G, s.n, s.offs, s.pal, s.idx, mab, se, out, A.APS_SYNC_PASS1 | route)
        A.aps_sync_noalloc(s.G, s.n, s.offs, s.pal, s.idx, mab, se, out, A.APS_SYNC_PASS2 | route)
    else:
        A.aps_sync_noalloc(s.G, s.n, s.offs, s.pal, s.idx, mab, se, out, BOTH | route)
    return out, se, mab


def _same(tag, got, ref):
    out, se, mab = (t.cpu().numpy() for t in got)
    r_out, r_se, r_mab = (t.cpu().numpy() for t in ref)
    assert same_maxabs(mab, r_mab), f"{tag}: maxima"
    assert np.array_equal(se, r_se), f"{tag}: scale exponents"
    assert same_f32(out, r_out), f"{tag}: sums {first_diff(out, r_out)}"


@pytest.mark.parametrize("split", [False, True], ids=["one call", "passes apart"])
@pytest.mark.parametrize("route", list(ROUTES), ids=list(ROUTES))
def test_noalloc_equals_aps_sync(dev, route, split):
    """A large set (ResNet-50, W = 8: 73 MiB of the array's 96), then a
    smaller one (ResNet-20, W = 8), then the large one again."""
    flag = ROUTES[route]
    big = _Set("resnet50_w8", "1-5-2", dev)
    small = _Set("resnet20", "1-4-3", dev)
    assert A.aps_sync_workspace_bytes(big.n, big.L) <= A.APS_SYNC_SCRATCH_BYTES
    for s in (big, small, big):
        tag = f"{s.name} W={s.W} {route} {'passes apart' if split else 'one call'}"
        log("noalloc", tag)
        got = _noalloc(s, flag, split)
        ref = _with_workspace(s, flag)
        torch.cuda.synchronize()
        _same(tag, got, ref)
    # the small set against the oracle as well
    G = small.G.cpu().numpy()
    opal = [ofmt(f) for f in small.pal]
    o_mab = O.layer_maxabs(G, small.n, small.gs.offsets)
    o_se = O.layer_scales(o_mab, small.W, opal)
    o_out = O.sim_reduce(G, small.n, small.gs.offsets, o_se, opal)
    out, se, mab = _noalloc(small, flag, split)
    torch.cuda.synchronize()
    assert same_maxabs(mab.cpu().numpy(), o_mab)
    assert np.array_equal(se.cpu().numpy(), o_se)
    assert same_f32(out.cpu().numpy(), o_out), first_diff(out.cpu().numpy(), o_out)
    del big, small
    torch.cuda.empty_cache()


def test_noalloc_hybrid_palette_and_w256(dev):
    """A two-format palette (its mixed chunks) and the 2-byte sums of the
    one-pass route at W = 256, two calls in a row, the second smaller."""
    for name, palette, W in (("resnet20", "1-5-2", 256), ("mlp", "1-4-3", 2)):
        gs = WL.generate(name, palette, device=dev, W=W)
        s = _Set.__new__(_Set)
        s.name, s.gs, s.G, s.n, s.W, s.L = f"{name} {palette}", gs, gs.G, gs.n, gs.W, len(gs.sizes)
        s.offs = torch.from_numpy(gs.offsets).to(dev)
        # every other layer in a second 8-bit format
        first = [A.Format(p.e, p.m, p.bias) for p in gs.palette]
        s.pal = first + [A.Format(4, 3) if first[0] == A.Format(5, 2) else A.Format(5, 2)]
        s.idx = torch.from_numpy((np.arange(s.L) % 2).astype(np.uint8)).to(dev)
        for route, flag in ROUTES.items():
            tag = f"{s.name} W={W} mixed palette {route}"
            log("noalloc", tag)
            got = _noalloc(s, flag, False)
            ref = _with_workspace(s, flag)
            torch.cuda.synchronize()
            _same(tag, got, ref)

