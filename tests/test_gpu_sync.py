"""GPU parity of aps_sync, one whole APS synchronisation per call, against
the CPU oracle.

aps_sync must return exactly what the oracle's max-abs, scales (N = W) and
rounded W-worker sum give (Algorithm 1 with the low-precision accumulator of
Sec. 5), whichever route the library takes: the one-pass route (the sum
formed unscaled while the maxima are taken, then the elements whose inputs
reach the format's subnormal range recomputed through the scaled path), the
guessed-scale route (the scaled sum formed with exponents guessed from every
32nd worker, layers whose guess was wrong rerun), or two passes.  The cases put
inputs exactly at, just above and just below each layer's threshold
2^(emin - ft), in fp32's subnormal range, in layers with INF/NaN or with a
maximum near fp32's top, and make chunks with few and with many elements to
recompute, so that both repair routes run.  Worker counts span the three
modes of the one-pass route's pass 1: fewer than 64 workers (no per-element
bytes, whole 256-element groups rerun), 64 and more (per-element bytes), and
from 128 with m <= 7 (the sums kept in 2 bytes and widened in pass 2)."""
import time
import zlib

import numpy as np
import pytest
import torch

import oracle as O
from paper_1911_08907_amd import aps as A
from paper_1911_08907_amd import workloads as WL
from tests._util import first_diff, log, ofmt, same_f32, same_maxabs
from tests.sync_cases import LAYER_MAXIMA, threshold_values
from tests.test_gpu_parity import _layout, _oracle_maxabs_streamed, _sample_idx, _sampled_oracle, _values

pytestmark = pytest.mark.gpu

F = A.Format
CH = 1024
SPARSE_MAX = 16


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    A.lib()  # the HIP library must be there: no fallback
    return torch.device("cuda:0")


BYTES_MIN_W = 64  # the one-pass route keeps per-element bytes from this many workers on


def _flagged(ws, n, offs, W):
    """Elements the second pass recomputed (read back from the workspace).
    From BYTES_MIN_W workers on: exponent byte below the layer's threshold.
    Below: every element of a 256-element group whose wave minimum is below
    the largest threshold of its chunk's layers."""
    if n == 0:
        return np.zeros(0, bool)
    L = offs.size - 1
    up = lambda b: (b + 255) // 256 * 256
    C = (n + CH - 1) // CH
    t0 = up(CH * C) + up(4 * C)
    w = ws.cpu().numpy()
    thr = w[t0:t0 + 4 * L].view(np.int32)
    layer = np.searchsorted(offs, np.arange(n), side="right") - 1
    if W >= BYTES_MIN_W:
        return w[:n].astype(np.int32) < thr[layer]
    wmin = w[up(CH * C):up(CH * C) + 4 * C].astype(np.int32).reshape(C, 4)
    starts = np.arange(C) * CH
    i0, i1 = layer[starts], layer[np.minimum(starts + CH, n) - 1]
    th = thr[i0].copy()
    for c in np.nonzero(i1 > i0)[0]:
        th[c] = thr[i0[c]:i1[c] + 1].max()
    groups = wmin < th[:, None]   # a group past n is never read below
    return np.repeat(groups.reshape(-1), 256)[:n]


def _rerun_layers(ws, n, L):
    """Layers the guessed-scale route reran (read back from the workspace):
    threshold 1 where the guessed exponent differed."""
    up = lambda b: (b + 255) // 256 * 256
    C = (n + CH - 1) // CH
    t0 = up(CH * C) + up(4 * C)
    return ws.cpu().numpy()[t0:t0 + 4 * L].view(np.int32) != 0


def _layer_mask(layers, n, offs):
    return layers[np.searchsorted(offs, np.arange(n), side="right") - 1] if n else np.zeros(0, bool)


def sync_case(dev, G, n, offs, pal, fmt_idx=None, tag="", split=False, garbage=True, route=A.APS_SYNC_ONE_PASS):
    W, ld = G.shape
    L = offs.size - 1
    opal = [ofmt(f) for f in pal]
    G_t = torch.from_numpy(G).to(dev)
    offs_t = torch.from_numpy(offs).to(dev)
    idx_t = None if fmt_idx is None else torch.from_numpy(fmt_idx).to(dev)
    ws = torch.empty(A.aps_sync_workspace_bytes(n, L), dtype=torch.uint8, device=dev)
    if garbage:  # the workspace's contents on entry must not matter
        ws.copy_(torch.randint(0, 256, ws.shape, dtype=torch.uint8, device=dev))
    out = torch.full((max(n, 1),), float("nan"), dtype=torch.float32, device=dev)
    mab = torch.full((L,), -1, dtype=torch.int32, device=dev)
    se = torch.full((L,), 12345, dtype=torch.int32, device=dev)
    if split:
        A.aps_sync(G_t, n, offs_t, pal, idx_t, A.APS_SYNC_PASS1 | route, mab, se, out, ws)
        A.aps_sync(G_t, n, offs_t, pal, idx_t, A.APS_SYNC_PASS2 | route, mab, se, out, ws)
    else:
        A.aps_sync(G_t, n, offs_t, pal, idx_t, A.APS_SYNC_PASS1 | A.APS_SYNC_PASS2 | route, mab, se, out, ws)
    torch.cuda.synchronize()
    o_mab = O.layer_maxabs(G, n, offs)
    assert same_maxabs(mab.cpu().numpy(), o_mab), f"{tag} maxabs"
    o_se = O.layer_scales(o_mab, W, opal, fmt_idx)
    assert np.array_equal(se.cpu().numpy(), o_se), f"{tag} scales"
    o_out = O.sim_reduce(G, n, offs, o_se, opal, fmt_idx)
    g = out.cpu().numpy()[:n]
    assert same_f32(g, o_out), f"{tag} sum {first_diff(g, o_out)}"
    taken = A.aps_sync_route(W, n, pal, route)
    if taken == A.APS_SYNC_ROUTE_ONE_PASS:
        return _flagged(ws, n, offs, W)
    if taken == A.APS_SYNC_ROUTE_GUESS:
        return _layer_mask(_rerun_layers(ws, n, L), n, offs)
    return None


# ----------------------------------------------------------- edge layouts

FORMATS = [F(5, 2), F(4, 3), F(3, 0), F(2, 0), F(2, 1), F(3, 2), F(5, 10), F(8, 7), F(8, 0), F(6, 1),
           F(4, 3, 5), F(5, 2, 20), F(7, 5), F(5, 12), F(8, 23), F(3, 12),
           F(8, 7, 130), F(5, 10, 120), F(3, 0, 145), F(2, 1, 147)]  # the last four round in fp64
SIZES = [0, 1, 3, 5, 7, 1023, 1024, 1025, 2049, 0, 64, 13, 4095, 2, 3000]


@pytest.mark.parametrize("f", FORMATS, ids=str)
@pytest.mark.parametrize("kind", ["normal", "special", "tiny"])
def test_sync_edge_layouts(dev, f, kind):
    seed = zlib.crc32(f"sync/{f}/{kind}".encode())  # stable across interpreters
    rng = np.random.default_rng(seed)
    offs, n, ld = _layout(SIZES)
    for W in (1, 2, 4, 8, 16, 3, 13, 40, 256):
        G = _values(rng, W, ld, offs, kind)
        tag = f"{f} {kind} W={W} seed={seed}"
        log("case", tag)
        sync_case(dev, G, n, offs, [f], tag=tag, split=(W == 4))
        sync_case(dev, G, n, offs, [f], tag=tag + " guessed scales", route=A.APS_SYNC_GUESS, split=(W == 3))
        if W in (2, 8):
            sync_case(dev, G, n, offs, [f], tag=tag + " default route", route=0)
            sync_case(dev, G, n, offs, [f], tag=tag + " two passes", route=A.APS_SYNC_TWO_PASS, split=(W == 2))


@pytest.mark.parametrize("seed", range(4))
def test_sync_mixed_palette(dev, seed):
    rng = np.random.default_rng(300 + seed)
    pal_choices = [[F(5, 2), F(4, 3), F(3, 0), F(2, 1)], [F(5, 10), F(5, 2), F(8, 7)],
                   [F(5, 2), F(4, 3), F(6, 1), F(3, 4)], [F(8, 23), F(5, 2), F(3, 0)]]
    pal = pal_choices[seed]
    sizes = [int(v) for v in rng.choice([0, 1, 2, 3, 5, 17, 255, 1000, 1023, 1024, 1500, 4096], 40)]
    offs, n, ld = _layout(sizes)
    fmt_idx = rng.integers(0, len(pal), len(sizes)).astype(np.uint8)
    for W in (2, 8, 5, 256):  # 256: 2-byte pass-1 sums where every format has m <= 7
        for kind in ("normal", "special", "tiny"):
            G = _values(rng, W, ld, offs, kind)
            tag = f"mixed seed={seed} W={W} {kind}"
            log("case", tag)
            sync_case(dev, G, n, offs, pal, fmt_idx=fmt_idx, tag=tag)
            sync_case(dev, G, n, offs, pal, fmt_idx=fmt_idx, tag=tag + " guessed scales", route=A.APS_SYNC_GUESS)


def test_many_tiny_layers(dev):
    """70,000 layers of 0 to 5 elements: every chunk spans hundreds of layers,
    and the grids over the layers pass 65,535 blocks.  The five calls and
    aps_sync on every route, one format and a two-format palette."""
    from tests.test_gpu_parity import run_case

    seed = zlib.crc32(b"many-tiny-layers")
    rng = np.random.default_rng(seed)
    sizes = [int(v) for v in rng.integers(0, 6, 70000)]
    offs, n, ld = _layout(sizes)
    fmt_idx = rng.integers(0, 2, len(sizes)).astype(np.uint8)
    for W in (4, 64, 128):
        G = _values(rng, W, ld, offs, "normal")
        tag = f"L={len(sizes)} n={n} W={W} seed={seed}"
        log("case", tag)
        if W == 4:
            run_case(dev, G, n, offs, [F(5, 2)], mode="aps", tag=tag + " calls")
            run_case(dev, G, n, offs, [F(5, 2), F(4, 3)], fmt_idx=fmt_idx, mode="aps", tag=tag + " calls mixed")
        for route, name in ((A.APS_SYNC_ONE_PASS, "one pass"), (A.APS_SYNC_GUESS, "guessed scales"),
                            (A.APS_SYNC_TWO_PASS, "two passes")):
            sync_case(dev, G, n, offs, [F(5, 2)], tag=f"{tag} {name}", route=route)
            sync_case(dev, G, n, offs, [F(5, 2), F(4, 3)], fmt_idx=fmt_idx, tag=f"{tag} {name} mixed", route=route)


def test_eight_format_palette(dev):
    """A palette of the maximum 8 formats (4-, 8- and 16-bit codes, one GEN
    format), layers assigned at random: the five calls and aps_sync on every
    route; and the 8 byte-code formats alone, codes included."""
    from tests.test_gpu_parity import run_case

    seed = zlib.crc32(b"eight-formats")
    rng = np.random.default_rng(seed)
    mixed = [F(5, 2), F(4, 3), F(3, 0), F(2, 1), F(6, 1), F(5, 10), F(8, 7), F(5, 10, 120)]
    bytes8 = [F(5, 2), F(4, 3), F(6, 1), F(3, 4), F(2, 5), F(4, 3, 5), F(5, 2, 20), F(7, 0)]
    assert len(mixed) == len(bytes8) == A.APS_MAX_FORMATS
    sizes = [int(v) for v in rng.choice([0, 1, 3, 17, 255, 1000, 1024, 1500, 4096], 60)]
    offs, n, ld = _layout(sizes)
    for pal, name in ((mixed, "mixed classes"), (bytes8, "byte codes")):
        fmt_idx = rng.integers(0, len(pal), len(sizes)).astype(np.uint8)
        for W in (3, 8, 128):
            G = _values(rng, W, ld, offs, "normal")
            tag = f"8 formats ({name}) W={W} seed={seed}"
            log("case", tag)
            run_case(dev, G, n, offs, pal, fmt_idx=fmt_idx, mode="aps", tag=tag + " calls")
            run_case(dev, G, n, offs, pal, fmt_idx=fmt_idx, mode="raw", tag=tag + " calls raw")
            for route in (A.APS_SYNC_ONE_PASS, A.APS_SYNC_GUESS, A.APS_SYNC_TWO_PASS, 0):
                sync_case(dev, G, n, offs, pal, fmt_idx=fmt_idx, tag=f"{tag} route {route}", route=route)


def test_calls_from_several_threads_and_streams(dev):
    """The header's thread-safety: four host threads, each on a stream of its
    own with its own buffers, call aps_sync (one-pass and guessed-scale
    routes) and the two-pass calls on different sets at the same time; every
    result equals the oracle's."""
    import threading

    seed = zlib.crc32(b"threads")
    rng = np.random.default_rng(seed)
    offs, n, ld = _layout(SIZES)
    jobs = []
    for k in range(4):
        W = (8, 256, 64, 3)[k]
        G = _values(rng, W, ld, offs, "normal")
        o_mab = O.layer_maxabs(G, n, offs)
        o_se = O.layer_scales(o_mab, W, [ofmt(F(5, 2))])
        jobs.append((G, O.sim_reduce(G, n, offs, o_se, [ofmt(F(5, 2))]), o_se))
    results, errors = {}, []
    offs_t = torch.from_numpy(offs).to(dev)

    def work(k):
        try:
            G, _, _ = jobs[k]
            stream = torch.cuda.Stream(device=dev)
            with torch.cuda.stream(stream):
                G_t = torch.from_numpy(G).to(dev, non_blocking=False)
                outs = []
                for it in range(6):
                    route = (A.APS_SYNC_ONE_PASS, A.APS_SYNC_GUESS, A.APS_SYNC_TWO_PASS)[it % 3]
                    o, se, _, _ = A.aps_sync(G_t, n, offs_t, [F(5, 2)], None,
                                             A.APS_SYNC_PASS1 | A.APS_SYNC_PASS2 | route)
                    outs.append((o, se))
                stream.synchronize()
                results[k] = [(o.cpu().numpy(), se.cpu().numpy()) for o, se in outs]
        except Exception as e:  # reported in the main thread
            errors.append(f"thread {k}: {e!r}")

    threads = [threading.Thread(target=work, args=(k,)) for k in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for k, (G, o_out, o_se) in enumerate(jobs):
        for it, (g, se) in enumerate(results[k]):
            tag = f"thread {k} W={G.shape[0]} call {it} seed={seed}"
            assert np.array_equal(se, o_se), f"{tag} scales"
            assert same_f32(g[:n], o_out), f"{tag} sum {first_diff(g[:n], o_out)}"
    log(f"4 threads x 6 calls on their own streams: all equal the oracle's (seed={seed})")


def test_sync_empty_gradient(dev):
    offs = np.zeros(4, np.int64)
    G = np.zeros((4, 4), np.float32)
    for route in (A.APS_SYNC_ONE_PASS, A.APS_SYNC_GUESS, A.APS_SYNC_TWO_PASS, 0):
        sync_case(dev, G, 0, offs, [F(5, 2)], tag=f"empty route={route}", route=route)


# ------------------------------------------------- thresholds and repair

@pytest.mark.parametrize("f", [F(5, 2), F(4, 3), F(3, 0), F(2, 1), F(5, 10), F(8, 7), F(6, 1), F(4, 3, 5)], ids=str)
def test_sync_threshold_inputs(dev, f):
    rng = np.random.default_rng(500 + f.e * 16 + f.m)
    sizes = [1, 7, 1024, 3000, 2, 5000, 64, 1025]
    offs, n, ld = _layout(sizes)
    for W in (1, 2, 4, 8, 64, 256):
        # maxima spread from tiny (threshold below 2^-126) to near fp32's top
        # (W = 256 with m <= 7: pass 1 keeps 2-byte sums)
        G = threshold_values(rng, W, ld, offs, f, LAYER_MAXIMA)
        tag = f"{f} thresholds W={W}"
        log("case", tag)
        fl = sync_case(dev, G, n, offs, [f], tag=tag)
        assert fl is not None and fl.any(), "no element was recomputed: the case tests nothing"


def _chunk_counts(flagged):
    n = flagged.size
    nch = (n + CH - 1) // CH
    pad = np.zeros(nch * CH, bool)
    pad[:n] = flagged
    return pad.reshape(nch, CH).sum(1)


def test_sync_sparse_and_dense_repairs(dev):
    """Chunks with 1..16 elements to recompute (one wave each) and with more
    (the whole chunk again), in the same call; W = 512 also walks the
    casts in two batches of 256 workers.  At W = 8 pass 1 keeps no
    per-element bytes, and whole 256-element groups are rerun."""
    f = F(5, 2)
    for W in (8, 512):
        n = 40 * CH
        ld = n
        rng = np.random.default_rng(W)
        G = (rng.standard_normal((W, ld)) * 0.1).astype(np.float32)
        G[0, 0] = 1.0
        ft = O.scale_one(int(np.float32(1.0).view(np.uint32)), W, ofmt(f))
        T = np.float32(2.0 ** (1 - f.b - ft))
        G[np.abs(G) < 64 * T] = 64 * T   # nothing flagged by chance
        # chunk c gets c elements whose first worker's input is below the
        # threshold (a first term is never swamped)
        planted = np.zeros(n, bool)
        for c in range(40):
            cols = c * CH + rng.choice(CH, c, replace=False)
            G[0, cols] = T * np.float32(0.75) * np.where(rng.random(c) < 0.5, -1, 1)
            planted[cols] = True
        # and below-threshold inputs from worker 1 meeting a first term of
        # 0.5: swamped, so nothing to recompute there
        sw = rng.choice(np.nonzero(~planted & (np.arange(n) > 0))[0], 500, replace=False)
        G[0, sw] = np.float32(0.5)
        G[1, sw] = T * np.float32(0.5)
        offs = np.array([0, n], np.int64)
        fl = sync_case(dev, G, n, offs, [f], tag=f"sparse/dense W={W}")
        cnt = _chunk_counts(fl)
        if W >= BYTES_MIN_W:
            assert np.array_equal(cnt, np.arange(40)), cnt
            assert ((cnt > 0) & (cnt <= SPARSE_MAX)).any() and (cnt > SPARSE_MAX).any()
        else:  # whole 256-element groups: every planted element among them, none in chunk 0
            assert fl[planted].all() and cnt[0] == 0, cnt


def test_sync_unsafe_layers(dev):
    """Layers whose max is INF or NaN, whose N * ghat overflows fp32, or
    exceeds 2^127: recomputed whole, through the scaled path."""
    f = F(5, 2)
    W = 4
    sizes = [300, 300, 300, 300, 300, 2000]
    offs, n, ld = _layout(sizes)
    rng = np.random.default_rng(9)
    G = (rng.standard_normal((W, ld)) * 1e-3).astype(np.float32)
    G[2, 10] = np.inf                       # layer 0: INF
    G[1, 310] = np.nan                      # layer 1: NaN
    with np.errstate(over="ignore"):
        G[:, 600:900] *= np.float32(3e38 / 4e-3)  # layer 2: N * ghat = INF
    G[0, 905] = np.float32(5e37)            # layer 3: N * ghat = 2e38, finite but above 2^127
    G[1, 906] = np.float32(-5e37)
    G[:, n:] = np.nan
    fl = sync_case(dev, G, n, offs, [f], tag="unsafe layers")
    assert fl[:1200].all()


def _guess_model(G, n, offs, W, f, stride=32):
    """The guessed exponents as the guessed-scale route defines them: the
    max over workers 0, 32, 64, ... (rows of them, n_s = rows * layer size
    values); t = fl32(N * max) raised by the expected growth of a normal
    sample's max, sqrt(1 + ln(N / rows) / ln max(n_s, 2)), where that stays
    finite; exponent emax - ceil(log2 t); 0 for a zero, INF or NaN max."""
    rows = (W + stride - 1) // stride
    ms = O.layer_maxabs(G[::stride], n, offs).view(np.float32)
    sizes = np.diff(offs)
    out = np.zeros(ms.size, np.int64)
    for i, m in enumerate(ms):
        if not (np.isfinite(m) and m > 0):
            continue
        t = np.float32(np.float32(W) * m)
        if not np.isfinite(t):
            continue
        grow = np.sqrt(1.0 + np.log(W / rows) / np.log(max(sizes[i] * rows, 2)))
        tn = np.float32(t * np.float32(grow))
        if np.isfinite(tn):
            t = tn
        fr, e = np.frexp(np.float64(t))
        out[i] = f.emax - (e - 1 if fr == 0.5 else e)
    return out


def test_sync_guess_reruns(dev):
    """The guessed-scale route with W = 40 (sampled workers 0 and 32, a
    300-element layer's max taken 1.21 times larger): layers whose guess is
    right (pass-1 sums kept) and wrong (rerun) of every kind: the max in an
    unsampled worker, a sampled max that the growth factor takes into the
    next binade with and without the full max getting there, INF outside the
    sample, NaN inside it, zeros, a max only outside the sample.  Sums
    against the oracle; the rerun layers against the guess rule."""
    f = F(4, 3)
    W = 40
    P = np.float32(4.0 / W)  # N * ghat = 4 * (this multiple of P)
    sizes = [300, 3000, 300, 300, 5000, 300, 300, 300, 1, 700, 2500, 300]
    offs, n, ld = _layout(sizes)
    rng = np.random.default_rng(40)
    G = (rng.standard_normal((W, ld)) * 0.01).astype(np.float32)
    G[:, n:] = np.nan
    lo = lambda i: int(offs[i])
    for i in range(4):
        G[:, lo(i):lo(i + 1)] = np.clip(G[:, lo(i):lo(i + 1)], -0.05, 0.05)
    G[32, lo(0) + 7] = 0.75 * P                    # 0: max sampled; 3.0 * 1.21 < 4: right
    G[0, lo(1) + 9] = 0.75 * P
    G[5, lo(1) + 2000] = 3.0 * P                    # 1: max outside the sample: wrong
    G[32, lo(2) + 1] = -0.9 * P                     # 2: 3.6 * 1.21 > 4, the full max stays below: wrong
    G[32, lo(3) + 3] = 0.9 * P
    G[7, lo(3) + 4] = 1.2 * P                       # 3: ... and the full max gets there: right
    G[9, lo(4) + 4321] = np.inf                     # 4: INF outside the sample: wrong
    G[0, lo(5) + 5] = np.nan                        # 5: NaN in the sample: right (exponent 0 both ways)
    G[:, lo(6):lo(7)] = 0.0                         # 6: all zero: right
    G[::32, lo(7):lo(8)] = 0.0                      # 7: zero in the sample: wrong
    G[:, lo(8)] = 0.0
    G[39, lo(8)] = 1e-3                             # 8: one element, only worker 39: wrong
    guess = _guess_model(G, n, offs, W, f)
    o_se = O.layer_scales(O.layer_maxabs(G, n, offs), W, ofmt(f))
    want = guess != o_se
    assert list(np.nonzero(want)[0][:5]) == [1, 2, 4, 7, 8], want
    assert not want[[0, 3, 5, 6]].any()
    for split in (False, True):
        rerun = sync_case(dev, G, n, offs, [f], tag=f"guess reruns split={split}", route=A.APS_SYNC_GUESS,
                          split=split)
        got = rerun[offs[:-1][np.array(sizes) > 0]]
        assert np.array_equal(got, want[np.array(sizes) > 0]), (got, want)


# --------------------------------------------------- paper-shaped sets

@pytest.mark.parametrize("name,palette", [("mlp", "1-4-3"), ("resnet20", "1-5-2"), ("resnet20", "1-4-3"),
                                          ("resnet20", "1-3-0")])
def test_sync_config_full(dev, name, palette):
    gs = WL.generate(name, palette, device="cpu")
    pal = [A.Format(p.e, p.m, p.bias) for p in gs.palette]
    fl = sync_case(dev, gs.G.numpy(), gs.n, gs.offsets, pal, fmt_idx=gs.fmt_idx, tag=f"{name} {palette}")
    log(name, palette, "recomputed", int(fl.sum()), "of", gs.n)
    fl = sync_case(dev, gs.G.numpy(), gs.n, gs.offsets, pal, fmt_idx=gs.fmt_idx, tag=f"{name} {palette} guessed",
                   route=A.APS_SYNC_GUESS)
    log(name, palette, "guessed scales: rerun", int(fl.sum()), "of", gs.n)


@pytest.mark.parametrize("name,palette", [("resnet50_w8", "1-5-2"), ("resnet50_w256", "1-5-2"),
                                          ("resnet50_w256", "1-4-3"), ("bert_large", "hybrid")])
def test_sync_config_large(dev, name, palette):
    """Full sizes: maxima and scales against the oracle in full, the sum
    against the two-pass kernels in full and against the oracle on sampled
    columns, the recomputed elements among them."""
    t0 = time.time()
    gs = WL.generate(name, palette, device=dev)
    G_t, W, n = gs.G, gs.W, gs.n
    pal = [A.Format(p.e, p.m, p.bias) for p in gs.palette]
    opal = [ofmt(f) for f in pal]
    offs_t = torch.from_numpy(gs.offsets).to(dev)
    idx_t = None if gs.fmt_idx is None else torch.from_numpy(gs.fmt_idx).to(dev)
    route = A.APS_SYNC_ONE_PASS   # the one-pass kernels at full size, also where the default would not take them
    out, se, mab, ws = A.aps_sync(G_t, n, offs_t, pal, idx_t, A.APS_SYNC_PASS1 | A.APS_SYNC_PASS2 | route)
    ref, se2, mab2 = A.aps_step(G_t, n, offs_t, pal, idx_t)
    dflt, _, _, _ = A.aps_sync(G_t, n, offs_t, pal, idx_t)
    gsd, gse, gmab, gws = A.aps_sync(G_t, n, offs_t, pal, idx_t, A.APS_SYNC_PASS1 | A.APS_SYNC_PASS2 | A.APS_SYNC_GUESS)
    torch.cuda.synchronize()
    assert torch.equal(gsd.view(torch.int32), ref.view(torch.int32)), "guessed-scale vs two-pass sum"
    assert torch.equal(gse, se2) and torch.equal(gmab, mab2), "guessed-scale scales / maxima"
    rr = _rerun_layers(gws, n, len(gs.sizes))
    log(name, palette, "guessed scales: rerun", int(rr.sum()), "layers,",
        int(np.array(gs.sizes)[rr].sum()), "of", n, "elements")
    del gsd, gws
    log(name, palette, "gpu done", f"{time.time() - t0:.1f}s")
    o_mab = _oracle_maxabs_streamed(G_t, gs)
    assert same_maxabs(mab.cpu().numpy(), o_mab), "maxabs"
    o_se = O.layer_scales(o_mab, W, opal, gs.fmt_idx)
    assert np.array_equal(se.cpu().numpy(), o_se), "scales"
    assert torch.equal(out.view(torch.int32), ref.view(torch.int32)), "one-pass vs two-pass sum"
    assert torch.equal(dflt.view(torch.int32), ref.view(torch.int32)), "default route vs two-pass sum"
    fl = _flagged(ws, n, gs.offsets, W)
    log(name, palette, "recomputed", int(fl.sum()), "of", n, f"{time.time() - t0:.1f}s")
    rng = np.random.default_rng(11)
    if name == "resnet50_w8":
        G = G_t.cpu().numpy()
        o_out = O.sim_reduce(G, n, gs.offsets, o_se, opal, gs.fmt_idx)
        g = out.cpu().numpy()
        assert same_f32(g, o_out), first_diff(g, o_out)
    else:
        idx = _sample_idx(rng, gs.offsets, n)
        fidx = np.nonzero(fl)[0]
        if fidx.size:
            idx = np.unique(np.concatenate([idx, rng.choice(fidx, min(fidx.size, 4000), replace=False)]))
        o_s = _sampled_oracle(G_t, gs, pal, idx, o_se, gs.fmt_idx, W)
        g = out[torch.from_numpy(idx).to(dev)].cpu().numpy()
        assert same_f32(g, o_s), first_diff(g, o_s)
        log("sampled parity on", idx.size, "columns,", int(fl[idx].sum()), "of them recomputed")
    assert bool(torch.isfinite(out).all())
    del G_t, gs
    torch.cuda.empty_cache()


# --------------------------------------------------------- maximum sizes

class _Set:
    """The fields of a generated gradient set the sampling helpers read."""

    def __init__(self, G_t, offsets):
        self.G, self.offsets = G_t, offsets
        self.W, self.n = G_t.shape[0], int(offsets[-1])


def test_sync_maximum_elements(dev):
    """n = APS_MAX_ELEMS (2^30 elements per worker), W = 2: maxima and scales
    in full, the sum on sampled columns (layer edges, chunk edges, both ends,
    random), both routes."""
    n = 1 << 30
    sizes = [1, 1000, (1 << 29) - 1001, 7, (1 << 29) - 7]
    offs = np.zeros(len(sizes) + 1, np.int64)
    offs[1:] = np.cumsum(sizes)
    assert offs[-1] == n
    g = torch.Generator(device=dev).manual_seed(1911)
    G_t = torch.randn((2, n), generator=g, device=dev) * 1e-3
    G_t[:, 1:1001] *= 1e-30
    offs_t = torch.from_numpy(offs).to(dev)
    pal = [F(5, 2)]
    t0 = time.time()
    out, se, mab, _ = A.aps_sync(G_t, n, offs_t, pal, None, A.APS_SYNC_PASS1 | A.APS_SYNC_PASS2 | A.APS_SYNC_ONE_PASS)
    out2, _, _, _ = A.aps_sync(G_t, n, offs_t, pal, None, A.APS_SYNC_PASS1 | A.APS_SYNC_PASS2 | A.APS_SYNC_TWO_PASS)
    out3, se3, _, _ = A.aps_sync(G_t, n, offs_t, pal, None, A.APS_SYNC_PASS1 | A.APS_SYNC_PASS2 | A.APS_SYNC_GUESS)
    torch.cuda.synchronize()
    log("n = 2^30 sync done", f"{time.time() - t0:.1f}s")
    assert torch.equal(out3.view(torch.int32), out2.view(torch.int32)), "guessed scales vs two passes"
    assert torch.equal(se3, se)
    del out3
    gs = _Set(G_t, offs)
    o_mab = _oracle_maxabs_streamed(G_t, gs, rows=1)
    assert same_maxabs(mab.cpu().numpy(), o_mab), "maxabs"
    o_se = O.layer_scales(o_mab, 2, [ofmt(f) for f in pal])
    assert np.array_equal(se.cpu().numpy(), o_se), "scales"
    assert torch.equal(out.view(torch.int32), out2.view(torch.int32)), "one pass vs two passes"
    idx = _sample_idx(np.random.default_rng(5), offs, n)
    o_s = _sampled_oracle(G_t, gs, pal, idx, o_se, None, 2)
    gv = out[torch.from_numpy(idx).to(dev)].cpu().numpy()
    assert same_f32(gv, o_s), first_diff(gv, o_s)
    del G_t, out, out2
    torch.cuda.empty_cache()


@pytest.mark.parametrize("W", [1 << 20, 1 << 24])
def test_sync_maximum_workers(dev, W):
    """W up to APS_MAX_WORKERS (2^24) on a 5-element gradient: the default
    route and the one-pass route, against the oracle in full."""
    n, ld = 5, 8
    offs = np.array([0, 2, 5], np.int64)
    rng = np.random.default_rng(W)
    G = (rng.standard_normal((W, ld)) * 1e-2).astype(np.float32)
    G[:, n:] = np.nan
    routes = [0] if W == 1 << 24 else [0, A.APS_SYNC_ONE_PASS, A.APS_SYNC_GUESS]
    for route in routes:
        t0 = time.time()
        sync_case(dev, G, n, offs, [F(5, 2)], tag=f"W={W} route={route}", route=route, garbage=False)
        log("W", W, "route", route, f"{time.time() - t0:.1f}s")


def test_sync_short_last_chunk_keeps_the_previous_chunks_bytes(dev):
    """A block that owns several chunks, the last of them short (300
    elements, so two of its waves hold no element): the chunk before it keeps
    its per-wave bytes, and its flagged elements in those waves' ranges are
    recomputed.  With W = 2 the launch has 8192 blocks, so 16385 chunks give
    two or three per block."""
    f = F(5, 2)
    W = 2
    n = 16384 * CH + 300
    ld = (n + 63) // 64 * 64
    g = torch.Generator(device=dev).manual_seed(7)
    G_t = torch.randn((W, ld), generator=g, device=dev) * 0.1
    G_t[0, 0] = 1.0
    ft = O.scale_one(int(np.float32(1.0).view(np.uint32)), W, ofmt(f))
    T = float(2.0 ** (1 - f.b - ft))
    G_t[G_t.abs() < 64 * T] = 64 * T                 # nothing below the threshold by chance
    c = 16383                                         # the chunk before the short last one
    # flagged elements of chunk c only in its waves 2 and 3 (elements 512..1023):
    # were their per-wave bytes lost, nothing would list the chunk
    planted = np.array([100 * CH + 5, c * CH + 600, c * CH + 900, c * CH + 1023, 16384 * CH + 10, 16384 * CH + 299])
    pt = torch.from_numpy(planted).to(dev)
    G_t[0, pt] = 0.6 * T                              # casts to 0.5 T scaled, 0.625 T unscaled
    G_t[1, pt] = 0.0
    offs = np.array([0, n], np.int64)
    offs_t = torch.from_numpy(offs).to(dev)
    out, se, mab, ws = A.aps_sync(G_t, n, offs_t, [f], None, A.APS_SYNC_PASS1 | A.APS_SYNC_PASS2 | A.APS_SYNC_ONE_PASS)
    torch.cuda.synchronize()
    fl = _flagged(ws, n, offs, W)
    assert fl[planted].all()
    gs = _Set(G_t[:, :n], offs)
    o_se = O.layer_scales(O.layer_maxabs(G_t.cpu().numpy(), n, offs), W, ofmt(f))
    assert np.array_equal(se.cpu().numpy(), o_se)
    idx = np.unique(np.concatenate([planted, _sample_idx(np.random.default_rng(3), offs, n)]))
    o_s = _sampled_oracle(G_t, gs, [f], idx, o_se, None, W)
    gv = out[torch.from_numpy(idx).to(dev)].cpu().numpy()
    assert same_f32(gv, o_s), first_diff(gv, o_s)


@pytest.mark.parametrize("route,W", [(A.APS_SYNC_ONE_PASS, 8), (A.APS_SYNC_TWO_PASS, 8), (A.APS_SYNC_GUESS, 8),
                                     (A.APS_SYNC_ONE_PASS, 256)],
                         ids=["one_pass", "two_passes", "guessed_scales", "one_pass_two_byte_sums"])
def test_sync_hip_graph_replays(dev, route, W):
    """aps_sync enqueues kernels only (no memset, no allocation), so it can be
    captured in a HIP graph: three replays on new inputs, with eager work
    between them, each against the oracle.  At W = 256 the one-pass route
    keeps its sums in 2 bytes and widens them in pass 2."""
    gs = WL.generate("resnet20", "1-5-2", device=dev, W=W)
    W, n, L = gs.W, gs.n, len(gs.sizes)
    pal = [F(5, 2)]
    opal = [ofmt(f) for f in pal]
    offs_t = torch.from_numpy(gs.offsets).to(dev)
    G = gs.G.clone()
    mab = torch.empty(L, dtype=torch.int32, device=dev)
    se = torch.empty(L, dtype=torch.int32, device=dev)
    out = torch.empty(n, dtype=torch.float32, device=dev)
    ws = torch.empty(A.aps_sync_workspace_bytes(n, L), dtype=torch.uint8, device=dev)
    flags = A.APS_SYNC_PASS1 | A.APS_SYNC_PASS2 | route
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        A.aps_sync(G, n, offs_t, pal, None, flags, mab, se, out, ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        A.aps_sync(G, n, offs_t, pal, None, flags, mab, se, out, ws)
    gen = torch.Generator(device=dev).manual_seed(23)
    for trial in range(3):
        # new inputs in place: rescaled rows plus noise, some exact zeros
        G.mul_(2.0 ** (trial - 1)).add_(torch.randn(G.shape, generator=gen, device=dev) * 1e-6)
        G[:, ::97] = 0.0
        eager = torch.empty_like(out)
        A.aps_sync(G, n, offs_t, pal, None, A.APS_SYNC_PASS1 | A.APS_SYNC_PASS2 | A.APS_SYNC_TWO_PASS, out=eager)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        Gh = G.cpu().numpy()
        o_mab = O.layer_maxabs(Gh, n, gs.offsets)
        assert same_maxabs(mab.cpu().numpy(), o_mab), f"replay {trial} maxabs"
        o_se = O.layer_scales(o_mab, W, opal)
        assert np.array_equal(se.cpu().numpy(), o_se), f"replay {trial} scales"
        o_out = O.sim_reduce(Gh, n, gs.offsets, o_se, opal)
        g = out.cpu().numpy()
        assert same_f32(g, o_out), f"replay {trial} {first_diff(g, o_out)}"
        assert torch.equal(out.view(torch.int32), eager.view(torch.int32)), f"replay {trial} vs eager"
