#!/usr/bin/env python3
"""Benchmark of the APS gradient path on one MI355X.

A step is one APS synchronisation of W simulated workers over a synthetic,
HBM-resident gradient set (Algorithm 1 of arXiv 1911.08907): per-layer
max-abs, per-layer scale exponents, and scale / cast / rounded W-worker sum /
unscale, through one aps_sync call (pass 1 + pass 2).  On the one-pass route
pass 1 reads the W rows once and forms the sum unscaled; pass 2 computes the
scales and recomputes the few elements whose inputs reach the format's
subnormal range.  On the guessed-scale route (formats of narrow range at
large W) pass 1 forms the scaled sum with exponents guessed from every 32nd
worker; pass 2 reruns the layers whose guess was wrong.  The default workload is the ResNet-50-shaped set with
W = 256 workers (161 tensors, 25,557,032 elements per worker, 26.2 GB of fp32
worker gradients) in the 1-5-2 format.

Prints one JSON line: whole-step throughput (worker-gradient elements per
second), the dominant kernel's HBM roofline figures measured with HIP events
on the launch stream, the two-pass step (max-abs, scales, fused reduce) and
the other calls timed beside it, and the CPU oracle's throughput on a
bounded sample.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "APS gradient elements/s (quantize+W-way sim reduce) and % of HBM peak GB/s"
HBM_PEAK_GBPS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = sorted(glob.glob(os.path.join(ROOT, "paper_1911_08907_amd", "csrc", "*.hip"))
                        + glob.glob(os.path.join(ROOT, "paper_1911_08907_amd", "csrc", "*.hpp")))


def source_digest(paths=None) -> str:
    """Digest of the kernel sources' code (all of them, or the given files,
    relative to the repository): comments and whitespace are dropped, so a
    change to a comment does not count as a kernel change."""
    h = hashlib.sha256()
    for p in (KERNEL_SOURCES if paths is None else [os.path.join(ROOT, q) for q in paths]):
        with open(p) as fh:
            txt = fh.read()
        txt = re.sub(r"/\*.*?\*/", " ", txt, flags=re.S)
        txt = re.sub(r"//[^\n]*", " ", txt)
        h.update(" ".join(txt.split()).encode())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="resnet50_w256")
    ap.add_argument("--palette", default=None)
    ap.add_argument("--mode", choices=["aps", "raw"], default="aps")
    ap.add_argument("--gemm", action="store_true", help="time only aps_lp_gemm (BERT-large FFN shape)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-calls", action="store_true",
                    help="skip timing aps_quantize / aps_dequantize outside the step")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="CPU oracle time budget")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip timing the other workloads (and RAW mode) after the headline step")
    ap.add_argument("--other-steps", type=int, default=10, help="timed steps per other workload")
    ap.add_argument("--roundoff", action="store_true",
                    help="only run the group-size round-off study (Eq. 5) and print it")
    ap.add_argument("--ceilings", action="store_true",
                    help="only time the path's access patterns without arithmetic, and VALU issue rates")
    ap.add_argument("--probe", default=None, help="with --ceilings: run only the probes whose names start so")
    ap.add_argument("--copy-calibration", type=float, default=0.0, metavar="GIB",
                    help="only run device-to-device copies of this size (counter calibration)")
    return ap.parse_args()


def copy_calibration(gib: float, reps: int = 5) -> None:
    import torch
    nbytes = int(gib * (1 << 30))
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_per_dispatch": nbytes, "reps": reps}), flush=True)


# ------------------------------------------------------------- ceilings

def _probe_lib():
    import ctypes

    from paper_1911_08907_amd import build as B

    if not os.path.exists(B.PROBE_LIB):
        raise RuntimeError(f"{B.PROBE_LIB} is missing: run paper_1911_08907_amd.build.build() first")
    L = ctypes.CDLL(B.PROBE_LIB)
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    for name, args in {"probe_rows": [i32, P, i32, i64, i64, P, P, P, i32, P],
                       "probe_flat": [i32, P, i32, i64, i64, P, i32, P],
                       "probe_rowmajor": [i32, i32, P, i32, i64, i64, P, i32, P],
                       "probe_flatrow_bytes": [i32, P, i32, i64, i64, P, i64, i32, P],
                       "probe_copy": [P, P, i64, i32, P],
                       "probe_rows_wide": [i32, i32, i32, P, i32, i64, i64, P, P, i32, P],
                       "probe_read_flat": [P, i64, P, i32, P],
                       "probe_copy_ranges": [P, P, i64, i32, P],
                       "probe_widen": [i32, i32, P, P, i64, i32, P],
                       "probe_valu": [i32, P, i32, i32, P]}.items():
        fn = getattr(L, name)
        fn.restype = ctypes.c_int
        fn.argtypes = args
    L.probe_device_cus.restype = ctypes.c_int
    return L


ROW_MODES = {"read": 0, "sum_f32": 1, "sum_half": 2, "sum_bytes": 3, "row_bytes": 4, "row_f32": 5}
# probe op id, instructions per step of a chain
VALU_OPS = {"v_add_f32_e32": (0, 1), "v_mul_f32_e32": (1, 1), "v_and_b32_e32": (2, 1), "v_fma_f32": (3, 1),
            "v_add3_u32": (4, 1), "v_bfe_u32": (5, 1), "v_ldexp_f32": (6, 1), "v_and_or_b32": (7, 1),
            "v_subrev_f32_e32": (8, 1), "v_cmp_nle_f32_e32+v_cndmask_b32_e32 (VCC)": (9, 2),
            "v_cmp_nle_f32_e64+v_cndmask_b32_e64 (SGPR mask)": (10, 2), "v_rndne_f32_e32": (11, 1),
            "v_pk_add_f16": (12, 1), "v_pk_mul_f16": (13, 1), "v_cvt_pk_bf16_f32": (14, 1)}


def ceilings(only: str | None = None, reps: int = 5) -> dict:
    """The access patterns of the path's kernels with no arithmetic
    (libaps_probe.so), timed with HIP events on the launch stream (median of
    `reps`), and the VALU issue rate of single instructions.  Sizes are the
    workloads': the ResNet-50 set at W = 256 and W = 8, BERT-large at W = 8."""
    import torch

    L = _probe_lib()
    dev = torch.device("cuda:0")
    torch.cuda.init()
    cus = L.probe_device_cus()
    stream = lambda: torch.cuda.current_stream().cuda_stream  # noqa: E731
    ptr = lambda t: None if t is None else t.data_ptr()  # noqa: E731
    res = {"device_cus": cus, "patterns": {}, "valu": {}}

    def want(name):
        return not only or name.startswith(only)

    def group(prefix):  # some probe named prefix... is wanted
        return not only or prefix.startswith(only) or only.startswith(prefix)

    def timed(name, fn, nbytes, **info):
        if not want(name):
            return
        st = fn()
        if st != 0:
            raise RuntimeError(f"probe {name}: status {st}")
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        t = sorted(ts)[len(ts) // 2]
        res["patterns"][name] = {"ms": t, "bytes": nbytes, "TBps": nbytes / (t * 1e-3) / 1e12,
                                 "frac_of_8TBps": nbytes / (t * 1e-3) / 1e12 / 8.0, **info}
        print(f"# {name}: {t:.4f} ms, {nbytes / (t * 1e-3) / 1e12:.2f} TB/s", file=sys.stderr, flush=True)

    def rows(tag, W, n_full, modes, widths, wide=()):
        n = n_full // 1024 * 1024
        ld = (n_full + 255) // 256 * 256  # rows padded as the workloads pad them
        writes_rows = any(m in ("row_bytes", "row_f32") for m in modes)
        names = [f"rows_{m}_{tag}_{b}percu" for m in modes for b in widths]
        names += [f"rows_wide{x}r{r}_{m}_{tag}_{b}percu" for x, r, m in wide for b in widths]
        if writes_rows:
            names += [f"{k}_{o}_{tag}" for k in ("flat", "rowmajor") for o in ("bytes", "f32")]
            names += [f"rowmajor_{o}_{g}inflight_{tag}" for o in ("bytes", "f32") for g in (1, 4, 8)]
            names += [f"flatrow_bytes_{k}_{tag}" for k in ("4B", "16B")]
        if only and not any(nm.startswith(only) or only.startswith(nm) for nm in names):
            return
        G = torch.zeros((W, ld), dtype=torch.float32, device=dev)
        out = torch.empty(n, dtype=torch.float32, device=dev)
        byt = torch.empty(n, dtype=torch.uint8, device=dev)
        half = torch.empty(n, dtype=torch.int16, device=dev)
        for m in modes:
            if not any(want(f"rows_{m}_{tag}_{b}percu") for b in widths):
                continue
            extra = {"read": 0, "sum_f32": 4, "sum_half": 2, "sum_bytes": 5, "row_bytes": W, "row_f32": 4 * W}[m]
            dst_o, dst_b = out, byt
            if m == "row_bytes":
                dst_b = torch.empty((W, ld), dtype=torch.uint8, device=dev)
            if m == "row_f32":
                dst_o = torch.empty((W, ld), dtype=torch.float32, device=dev)
            for bpc in widths:
                timed(f"rows_{m}_{tag}_{bpc}percu",
                      lambda: L.probe_rows(ROW_MODES[m], ptr(G), W, ld, n, ptr(dst_o), ptr(dst_b), ptr(half), bpc,
                                           stream()),
                      4.0 * W * n + extra * n, W=W, n=n, blocks_per_cu=bpc)
            del dst_o, dst_b
            torch.cuda.empty_cache()
        # the same walk with chx chunks side by side per block step (each row read in runs of chx * 4 KB)
        for chx, r, m in wide:
            nw = n_full // (chx * 1024) * (chx * 1024)
            extra = {"read": 0, "sum_half": 2, "sum_f32": 4}[m]
            for bpc in widths:
                timed(f"rows_wide{chx}r{r}_{m}_{tag}_{bpc}percu",
                      lambda: L.probe_rows_wide(chx, r, {"read": 0, "sum_half": 1, "sum_f32": 2}[m], ptr(G), W, ld,
                                                nw, ptr(out), ptr(half), bpc, stream()),
                      4.0 * W * nw + extra * nw, W=W, n=nw, chunks_per_step=chx, rows_per_set=r, blocks_per_cu=bpc)
        if writes_rows:
            for outb in (1, 4):
                kind = "bytes" if outb == 1 else "f32"
                if not (group(f"flat_{kind}_{tag}") or group(f"rowmajor_{kind}_")):
                    continue
                dst = torch.empty((W, ld * outb), dtype=torch.uint8, device=dev)
                for bpc in (8, 16, 32):
                    timed(f"flat_{kind}_{tag}_{bpc}percu",
                          lambda: L.probe_flat(outb, ptr(G), W, ld, n // 4096 * 4096, ptr(dst), bpc, stream()),
                          (4.0 + outb) * W * (n // 4096 * 4096), W=W, n=n // 4096 * 4096, blocks_per_cu=bpc)
                for g in (1, 4, 8):
                    for bpc in (8, 16):
                        timed(f"rowmajor_{kind}_{g}inflight_{tag}_{bpc}percu",
                              lambda: L.probe_rowmajor(outb, g, ptr(G), W, ld, n, ptr(dst), bpc, stream()),
                              (4.0 + outb) * W * n, W=W, n=n, chunks_in_flight=g, blocks_per_cu=bpc)
                del dst
                torch.cuda.empty_cache()
            if group(f"flatrow_bytes_"):
                # a coalesced flat walk: 4 chunks of one row per block step, code bytes stored 4 or 16 per lane
                nf = n // 4096 * 4096
                dst = torch.empty((W, ld), dtype=torch.uint8, device=dev)
                for staged, kname in ((0, "4B"), (1, "16B")):
                    for bpc in (8, 16, 32):
                        timed(f"flatrow_bytes_{kname}_{tag}_{bpc}percu",
                              lambda: L.probe_flatrow_bytes(staged, ptr(G), W, ld, nf, ptr(dst), ld, bpc, stream()),
                              5.0 * W * nf, W=W, n=nf, blocks_per_cu=bpc)
                del dst
                torch.cuda.empty_cache()
        del G, out, byt, half
        torch.cuda.empty_cache()

    n50, n_bert = 25557032, 335141888
    rows("resnet50_w256", 256, n50, ["read", "sum_f32", "sum_half", "sum_bytes", "row_bytes", "row_f32"], (16, 24),
         wide=[(2, 2, "read"), (4, 2, "read"), (2, 2, "sum_half"), (4, 2, "sum_half")])
    rows("resnet50_w8", 8, n50, ["read", "sum_f32", "sum_bytes", "row_bytes"], (32, 64),
         wide=[(2, 4, "sum_f32"), (4, 2, "sum_f32")])
    bert_wide = min(512, (n_bert // 1024) * 2 // (cus * 5))
    rows("bert_large", 8, n_bert, ["read", "sum_f32", "sum_bytes"], (32, bert_wide),
         wide=[(2, 4, "sum_f32"), (4, 2, "sum_f32")])
    if group("read_flat_8GiB"):
        n = 1 << 31  # 8 GiB
        a = torch.zeros(n, dtype=torch.float32, device=dev)
        sink = torch.empty(256, dtype=torch.float32, device=dev)
        for bpc in (8, 16, 32):
            timed(f"read_flat_8GiB_{bpc}percu", lambda: L.probe_read_flat(ptr(a), n, ptr(sink), bpc, stream()),
                  4.0 * n, n=n, blocks_per_cu=bpc)
        del a, sink
        torch.cuda.empty_cache()
    if group("copy_2GiB") or group("copy_ranges_2GiB"):
        n = 1 << 29  # 2 GiB
        a = torch.zeros(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for bpc in (8, 32):
            timed(f"copy_2GiB_{bpc}percu", lambda: L.probe_copy(ptr(a), ptr(b), n, bpc, stream()), 8.0 * n,
                  n=n, blocks_per_cu=bpc)
        for bpc in (8, 16, 32):
            timed(f"copy_ranges_2GiB_{bpc}percu", lambda: L.probe_copy_ranges(ptr(a), ptr(b), n, bpc, stream()),
                  8.0 * n, n=n, blocks_per_cu=bpc)
        del a, b
        torch.cuda.empty_cache()
    if group("widen_"):
        n = n50 // 16 * 16
        src = torch.zeros(2 * n, dtype=torch.uint8, device=dev)
        dst = torch.empty(n, dtype=torch.float32, device=dev)
        for ib, per in ((1, 4), (1, 16), (2, 16)):
            for bpc in (8, 32):
                timed(f"widen_{ib}B_{per}perthread_resnet50_{bpc}percu",
                      lambda: L.probe_widen(ib, per, ptr(src), ptr(dst), n, bpc, stream()), (ib + 4.0) * n,
                      n=n, in_bytes=ib, per_thread=per, blocks_per_cu=bpc)
        del src, dst
        torch.cuda.empty_cache()
    if group("valu_"):
        sink = torch.empty(256, dtype=torch.float32, device=dev)
        iters, bpc = 2048, 16
        blocks = cus * bpc
        for name, (op, per_step) in VALU_OPS.items():
            if not want(f"valu_{name}"):
                continue
            L.probe_valu(op, ptr(sink), bpc, iters, stream())
            torch.cuda.synchronize()
            ts = []
            for _ in range(reps):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                L.probe_valu(op, ptr(sink), bpc, iters, stream())
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1))
            t = sorted(ts)[len(ts) // 2]
            lane_instr = blocks * 256.0 * iters * 64 * per_step
            rate = lane_instr / (t * 1e-3)
            res["valu"][name] = {"ms": t, "lane_instr_per_s": rate,
                                 "lanes_per_clk_per_cu_at_2.4GHz": rate / cus / 2.4e9,
                                 "frac_of_78.6T": rate / (VALU_PEAK_T * 1e12)}
            print(f"# {name}: {rate / cus / 2.4e9:.1f} lanes/clk/CU", file=sys.stderr, flush=True)
    return res


def traffic_from_profile(kernel: str, config: str, palette: str):
    """HBM bytes per launch of `kernel` from the committed counter summary,
    if it was taken on the current kernel source."""
    path = os.path.join(PROFILES, f"{kernel}_{config}_{palette}_counters.json")
    if not os.path.exists(path):
        return None, "no counter summary"
    with open(path) as fh:
        c = json.load(fh)
    # the digest covers the files the kernel is compiled from, as the summary lists them
    if c.get("source_digest") != source_digest(c.get("sources")):
        return None, "kernel changed since the counters were taken"
    fetch = c["fetch_kib_per_dispatch"] * 1024 * c["fetch_scale"]
    write = c["write_kib_per_dispatch"] * 1024 * c["write_scale"]
    return fetch + write, f"{os.path.basename(path)}"


def event_timed(fns, reps: int = 5):
    """Median over reps of the event-timed span of each callable in fns,
    run back to back on the current stream."""
    import torch

    for fn in fns:
        fn()
    torch.cuda.synchronize()
    spans = [[] for _ in fns]
    for _ in range(reps):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(fns) + 1)]
        ev[0].record()
        for k, fn in enumerate(fns):
            fn()
            ev[k + 1].record()
        torch.cuda.synchronize()
        for k in range(len(fns)):
            spans[k].append(ev[k].elapsed_time(ev[k + 1]))
    return [sorted(t)[len(t) // 2] for t in spans]


def two_pass_step(A, G, gs, pal, idx_t, offs_t, mab, se, out):
    """The step as three calls (max-abs, scales, fused reduce): two full
    reads of the W rows."""
    W, n = gs.W, gs.n
    t1, t2, t3 = event_timed([lambda: A.aps_layer_maxabs(G, n, offs_t, mab),
                              lambda: A.aps_layer_scales(mab, W, pal, idx_t, se),
                              lambda: A.aps_sim_reduce(G, n, offs_t, se, pal, idx_t, 0, out=out)])
    return {"ms": t1 + t2 + t3, "elements_per_s": W * n / ((t1 + t2 + t3) * 1e-3),
            "kernels_ms": {"k_maxabs": t1, "k_scales": t2, "k_sim_reduce": t3},
            "k_sim_reduce_GBps": (4.0 * W * n + 4.0 * n) / (t3 * 1e-3) / 1e9}


def other_calls(A, G, gs, pal, idx_t, offs_t, se, out, reps: int = 5):
    """Event-timed aps_quantize (codes out) and aps_dequantize (codes in) on
    the same set, outside the timed step; GB/s from their algorithmic bytes."""
    import torch

    bits = max(f.bits for f in pal)
    if len({A.code_bytes(8, f.bits) for f in pal}) != 1 or bits > 16:
        return {}
    W, n, ld = gs.W, gs.n, gs.ld
    row_bytes = A.code_bytes(ld, bits)
    codes = torch.empty(W * row_bytes, dtype=torch.uint8, device=G.device)
    rcodes = codes[:A.code_bytes(n, bits) + 16]
    res = {}

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return sorted(ts)[len(ts) // 2]

    cb = A.code_bytes(W * n, bits)
    t = timed(lambda: A.aps_quantize(G, n, offs_t, se, pal, idx_t, Q=None, codes=codes))
    res["quantize_to_codes"] = {"ms": t, "GBps": (4.0 * W * n + cb) / (t * 1e-3) / 1e9}
    if row_bytes % 16 == 0:
        # the W-worker sum over the codes themselves (the exchanged form)
        t = timed(lambda: A.aps_sim_reduce_codes(codes, W, ld, n, offs_t, se, pal, idx_t, 0, out=out))
        res["sim_reduce_codes"] = {"ms": t, "GBps": (A.code_bytes(n, bits) * W + 4.0 * n) / (t * 1e-3) / 1e9,
                                   "elements_per_s": W * n / (t * 1e-3)}
        if W >= 8:
            # one owner's share on an 8-GPU node: the 8 workers' code rows of
            # its n/8 elements (here rows 0..7 and elements [0, n/8), the
            # layer table cut there), reduced in worker order
            import numpy as np
            n8 = n // 8
            offs = offs_t.cpu().numpy()
            L8 = int(np.searchsorted(offs, n8, side="left"))
            offs8 = torch.from_numpy(np.append(offs[:L8], n8).astype(np.int64)).to(G.device)
            se8 = None if se is None else se[:L8].contiguous()
            idx8 = None if idx_t is None else idx_t[:L8].contiguous()
            out8 = out[:n8]
            t = timed(lambda: A.aps_sim_reduce_codes(codes[:8 * row_bytes], 8, ld, n8, offs8, se8, pal, idx8, 0,
                                                     out=out8))
            res["owner_reduce_codes_8gpu"] = {
                "shape": f"8 code rows x {n8} elements (one owner's n/8 slice on an 8-GPU node)",
                "ms": t, "GBps": (A.code_bytes(n8, bits) * 8 + 4.0 * n8) / (t * 1e-3) / 1e9}
    # summation orders of the hierarchical all-reduce and the Kahan accumulator (fp32 input)
    for name, k, acc in (("sim_reduce_ex_group16", 16, A.APS_ACC_SEQUENTIAL), ("sim_reduce_ex_ring", 1, A.APS_ACC_SEQUENTIAL),
                         ("sim_reduce_ex_kahan", None, A.APS_ACC_KAHAN)):
        if k is not None and W % k:
            continue
        t = timed(lambda: A.aps_sim_reduce_ex(G, n, offs_t, se, pal, idx_t, 0, group=k, accumulator=acc, out=out))
        res[name] = {"ms": t, "GBps": (4.0 * W * n + 4.0 * n) / (t * 1e-3) / 1e9, "elements_per_s": W * n / (t * 1e-3)}
    A.aps_sim_reduce(G, n, offs_t, se, pal, idx_t, A.APS_OUTPUT_SCALED, out=None, codes_out=rcodes)
    t = timed(lambda: A.aps_dequantize(None, rcodes, n, offs_t, se, pal, idx_t, out))
    res["dequantize_from_codes"] = {"ms": t, "GBps": (A.code_bytes(n, bits) + 4.0 * n) / (t * 1e-3) / 1e9}
    del codes
    return res


ROUNDOFF_GROUPS = (4, 8, 16, 32, 64, 1)


def round_off_error(grad_h, grad_l) -> float:
    """Eq. (5): the mean over the elements with grad_h != 0 of
    |(grad_h - grad_l) / grad_h|, in double (0 when every grad_h is 0).
    grad_h is the fp32 all-reduce, grad_l the low-precision one."""
    import numpy as np

    h = np.asarray(grad_h, np.float32).astype(np.float64)
    lo = np.asarray(grad_l, np.float32).astype(np.float64)
    nz = h != 0
    if not nz.any():
        return 0.0
    return float(np.mean(np.abs((h[nz] - lo[nz]) / h[nz])))


def roundoff_arrays(groups=ROUNDOFF_GROUPS):
    """The data of Sec. 4.2's round-off study on synthetic gradients: the
    first convolution's gradient (64x3x7x7) for W = 256 workers, reduced in
    fp32 (1-8-23, worker order) and in 1-5-2 with APS scales by hierarchical
    all-reduces of several group sizes (1 is the ring over all workers).  Two
    draws: the configs' recipe (workers independent, so their sum largely
    cancels) and correlated workers (a shared gradient plus per-worker noise
    of the same size, which is how data-parallel gradients relate).  Returns
    {draw: (G, scale_exp, grad_h, {group name: grad_l})}, host arrays."""
    import torch

    from paper_1911_08907_amd import aps as A
    from paper_1911_08907_amd import workloads as WL

    dev = torch.device("cuda:0")
    W, n = 256, 64 * 3 * 7 * 7
    ld = (n + 63) // 64 * 64
    offs_t = torch.tensor([0, n], dtype=torch.int64, device=dev)
    g = torch.Generator(device=dev)
    g.manual_seed(WL.BASE_SEED)
    s = 1e-3
    draws = {
        "independent": torch.randn(W, ld, generator=g, device=dev) * s,
        "correlated": (torch.randn(1, ld, generator=g, device=dev) + torch.randn(W, ld, generator=g, device=dev)) * s,
    }
    out = {}
    for name, G in draws.items():
        G[:, n:] = 0
        hi = torch.empty(n, dtype=torch.float32, device=dev)
        A.aps_sim_reduce(G, n, offs_t, None, [A.Format(8, 23)], None, 0, out=hi)
        _, se, _ = A.aps_step(G, n, offs_t, [A.Format(5, 2)])
        lo = {}
        for k in groups:
            t = torch.empty(n, dtype=torch.float32, device=dev)
            A.aps_sim_reduce_ex(G, n, offs_t, se, [A.Format(5, 2)], None, 0, group=k, out=t)
            lo["ring_256" if k == 1 else f"group_{k}"] = t
        torch.cuda.synchronize()
        out[name] = (G.cpu().numpy(), se.cpu().numpy(), hi.cpu().numpy(), {k: t.cpu().numpy() for k, t in lo.items()})
    return out


ROUNDOFF_STUDY = ("Eq.5 round-off error vs all-reduce group size, 64x3x7x7 gradient, W=256, "
                  "1-5-2 with APS scales, synthetic")


def roundoff_study(groups=ROUNDOFF_GROUPS) -> dict:
    """Eq. (5) for each draw and group size of roundoff_arrays."""
    return {name: {k: round_off_error(h, lo) for k, lo in lows.items()}
            for name, (_, _, h, lows) in roundoff_arrays(groups).items()}


def cpu_description() -> dict:
    """The host CPU as lscpu reports it (model, sockets, physical cores,
    logical CPUs), and the CPUs this process may run on."""
    import subprocess

    info = {}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
        for line in out.splitlines():
            k, _, v = line.partition(":")
            info[k.strip()] = v.strip()
    except (OSError, subprocess.SubprocessError):
        pass
    model = info.get("Model name")
    if not model:
        try:
            with open("/proc/cpuinfo") as fh:
                model = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), None)
        except OSError:
            model = None

    def num(key):
        try:
            return int(info[key])
        except (KeyError, ValueError):
            return None

    sockets, cores = num("Socket(s)"), num("Core(s) per socket")
    try:
        allowed = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        allowed = None
    return {"cpu_model": model or "unknown", "sockets": sockets,
            "physical_cores": sockets * cores if sockets and cores else None,
            "logical_cpus": num("CPU(s)"), "threads_per_core": num("Thread(s) per core"),
            "cpus_allowed": allowed}


def _omp_threads(k: int) -> bool:
    """Set the OpenMP thread count of this process (the oracle's runtime);
    False if the runtime cannot be reached."""
    import ctypes

    try:
        ctypes.CDLL("libgomp.so.1").omp_set_num_threads(int(k))
    except (OSError, AttributeError):
        return False
    return True


def cpu_baseline(G_t, gs, pal, budget_s: float, slice_cols: int = 65536, single_s: float = 3.0):
    """The CPU oracle on successive column slices (all W workers) of the same
    gradient set until the time budget is used: max-abs, scales and the
    rounded W-worker sum for each slice.  Run with all the OpenMP threads,
    then on one thread over a shorter budget."""
    import numpy as np

    import oracle as O

    opal = [O.Format(f.e, f.m, f.bias) for f in pal]
    W, n = gs.W, gs.n

    def run(budget):
        done, spent, start_col = 0, 0.0, 0
        while spent < budget and start_col < n:
            cols = min(slice_cols, n - start_col)
            Gs = G_t[:, start_col:start_col + cols].cpu().numpy()
            offs = gs.offsets
            lo = np.searchsorted(offs, start_col, side="right") - 1
            hi = np.searchsorted(offs, start_col + cols, side="left")
            sub = np.clip(offs[lo:hi + 1] - start_col, 0, cols).astype(np.int64)
            sub[0], sub[-1] = 0, cols
            fi = None if gs.fmt_idx is None else gs.fmt_idx[lo:hi]
            ldS = (cols + 3) // 4 * 4
            Gp = np.zeros((W, ldS), np.float32)
            Gp[:, :cols] = Gs
            t0 = time.perf_counter()
            mab = O.layer_maxabs(Gp, cols, sub)
            se = O.layer_scales(mab, W, opal, fi)
            O.sim_reduce(Gp, cols, sub, se, opal, fi)
            spent += time.perf_counter() - t0
            done += cols
            start_col += cols
        return done, spent

    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    O.lib()  # load the oracle (and its OpenMP runtime) before setting its thread count
    can_set = _omp_threads(threads)
    done, spent = run(budget_s)
    single = None
    if can_set and _omp_threads(1):
        done1, spent1 = run(single_s)
        _omp_threads(threads)
        single = (W * done1 / spent1, f"first {done1} elements x all {W} workers, {spent1:.1f} s")
    return {
        "value": W * done / spent,
        "unit": "elements/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"first {done} of {n} elements x all {W} workers, in {slice_cols}-element column slices "
                  f"(max-abs + scales + rounded W-worker sum), {spent:.1f} s",
        "single_thread_value": single[0] if single else None,
        "single_thread_sample": single[1] if single else "OpenMP runtime not reachable: not measured",
        **cpu_description(),
    }


# VALU peak: 256 CUs x 128 lanes/clk x 2.4 GHz = 78.6 T lane-instructions/s,
# the published 157.3 TFLOP/s fp32 vector rate counted one lane-instruction
# per FMA.
VALU_PEAK_T = 256 * 128 * 2.4e9 / 1e12
# Issue rates of the instructions of the GEMM kernels' k-loops, lanes per
# clock per CU at 2.4 GHz, measured by bench.py --ceilings (chains of one
# instruction, profiles/ceilings_patterns_and_valu.txt): two-operand adds,
# multiplies and ands issue at about 112-120; v_bfe_u32, v_add3_u32,
# v_rndne_f32 and the packed half-precision v_pk_add_f16 / v_pk_mul_f16
# (two lanes of work each) at about 62.
VALU_RATES = {"v_and_b32": 119.3, "v_add_f32": 112.7, "v_sub_f32": 118.5, "v_mul_f32": 116.6,
              "v_bfe_u32": 62.1, "v_add3_u32": 62.2, "v_rndne_f32": 62.7,
              "v_pk_add_f16": 62.2, "v_pk_mul_f16": 62.0, "v_cvt_pk_bf16_f32": 62.2,
              "v_lshlrev_b32": 115.0}  # the shift not probed: the two-operand forms' rate
# VALU instructions per multiply-accumulate of each k-loop, counted in the
# kernels' ISA (one loop iteration: 16 k-steps of the thread's 4 x 4 outputs).
#   k_lp_gemm_h (the accumulator is IEEE half): a packed multiply and a packed
#     add per two outputs; Kahan four packed adds.  The loop also issues 16
#     ds_read2_b64 (the operands from LDS).
#   k_lp_gemm, products on the accumulator's subnormal grid (1-5-2 inputs into
#     1-5-7): the product, its rint, the multiply into the working domain, the
#     add and its rounding (v_bfe_u32, v_add3_u32, v_and_b32); Kahan rounds four
#     adds.  The loop also issues 32 ds_read_b128.
#   k_lp_gemm, exact products into bfloat16 (1-5-2 inputs into 1-8-7: every
#     product fits and none is subnormal): the product, the add, and its
#     rounding by a packed conversion to bfloat16 for two chains
#     (v_cvt_pk_bf16_f32) and the two halves taken back (v_lshlrev_b32,
#     v_and_b32); Kahan rounds four adds so.
GEMM_LOOP_MIX = {
    "sequential": {"v_pk_mul_f16": 0.5, "v_pk_add_f16": 0.5},
    "kahan": {"v_pk_mul_f16": 0.5, "v_pk_add_f16": 2.0},
    "sequential_emulated": {"v_mul_f32": 2, "v_rndne_f32": 1, "v_add_f32": 1, "v_and_b32": 1, "v_bfe_u32": 1,
                            "v_add3_u32": 1},
    "kahan_emulated": {"v_mul_f32": 2, "v_rndne_f32": 1, "v_add_f32": 1, "v_sub_f32": 3, "v_and_b32": 4,
                       "v_bfe_u32": 4, "v_add3_u32": 4},
    "sequential_bf16": {"v_mul_f32": 1, "v_add_f32": 1, "v_cvt_pk_bf16_f32": 0.5, "v_lshlrev_b32": 0.5,
                        "v_and_b32": 0.5},
    "kahan_bf16": {"v_mul_f32": 1, "v_add_f32": 1, "v_sub_f32": 3, "v_cvt_pk_bf16_f32": 2, "v_lshlrev_b32": 2,
                   "v_and_b32": 2},
}
GEMM_SHAPE = (4096, 1024, 4096)  # BERT-large FFN up-projection at 8 x 512 tokens: M, K, N


def lp_gemm_calls(A, dev, reps: int = 5):
    """Event-timed aps_lp_gemm on the BERT-large FFN shape with 1-5-2 inputs:
    a 1-5-10 accumulator (IEEE half: k_lp_gemm_h), a 1-5-7 one and a
    bfloat16 one (emulated in fp32: k_lp_gemm), plain and Kahan; an ALU
    roofline from the VALU instructions each kernel issues per
    multiply-accumulate."""
    import torch

    M, K, N = GEMM_SHAPE
    g = torch.Generator(device=dev).manual_seed(1911)
    Am = torch.randn((M, K), generator=g, device=dev)
    Bm = torch.randn((K, N), generator=g, device=dev) * 0.02
    C = torch.empty((M, N), device=dev)
    fin = A.Format(5, 2)
    res = {"workload": f"bert_large_ffn M={M} K={K} N={N}", "in": str(fin)}
    cases = (("sequential", A.APS_ACC_SEQUENTIAL, A.Format(5, 10), "k_lp_gemm_h"),
             ("kahan", A.APS_ACC_KAHAN, A.Format(5, 10), "k_lp_gemm_h"),
             ("sequential_emulated", A.APS_ACC_SEQUENTIAL, A.Format(5, 7), "k_lp_gemm"),
             ("kahan_emulated", A.APS_ACC_KAHAN, A.Format(5, 7), "k_lp_gemm"),
             ("sequential_bf16", A.APS_ACC_SEQUENTIAL, A.Format(8, 7), "k_lp_gemm"),
             ("kahan_bf16", A.APS_ACC_KAHAN, A.Format(8, 7), "k_lp_gemm"))
    for name, acc, facc, kernel in cases:
        A.aps_lp_gemm(Am, Bm, fin, facc, acc, C=C)
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            A.aps_lp_gemm(Am, Bm, fin, facc, acc, C=C)
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        t = sorted(ts)[len(ts) // 2]
        macs = float(M) * N * K
        mix = GEMM_LOOP_MIX[name]
        instr = float(sum(mix.values()))
        achieved = macs * instr / (t * 1e-3) / 1e12
        # the mix's own ceiling: every CU issuing the loop's instructions at
        # their measured rates, back to back
        clk_per_lane_mac = sum(k / VALU_RATES[op] for op, k in mix.items())
        ceiling = 256 * 2.4e9 / clk_per_lane_mac
        res[name] = {"acc": str(facc), "kernel": kernel, "ms": t, "MAC_per_s": macs / (t * 1e-3),
                     "roofline": {"bound": "alu", "achieved": achieved, "peak": VALU_PEAK_T,
                                  "unit": "T VALU lane-instructions/s", "frac": achieved / VALU_PEAK_T,
                                  "valu_per_mac": instr, "mix_ceiling_MAC_per_s": ceiling,
                                  "frac_of_mix_ceiling": macs / (t * 1e-3) / ceiling}}
    return res


def measure_step(A, gs, pal, idx_t, offs_t, mode: str, steps: int, warmup: int, graph: bool = False,
                 loops: int = 1) -> dict:
    """Time `steps` APS synchronisations of a gradient set after `warmup`
    untimed ones: aps_sync's pass 1 and pass 2 as two calls (APS mode), or
    the reduce with every exponent 0 (RAW mode, casting without APS).  The
    step time is wall-clock over steps run back to back; the pass spans come
    from as many further steps with HIP events around each pass on the
    launch stream.  With loops > 1 the back-to-back run is repeated and the
    median of its per-step times is kept (a host hiccup of a few ms in one
    short run would otherwise weigh on the figure).  Returns the step time,
    the pass times, the route and the dominant kernel's roofline figures,
    plus the device arrays the step wrote."""
    import torch

    dev = gs.G.device
    G, W, n, L = gs.G, gs.W, gs.n, len(gs.sizes)
    mab = torch.empty(L, dtype=torch.int32, device=dev)
    se = torch.empty(L, dtype=torch.int32, device=dev)
    out = torch.empty(n, dtype=torch.float32, device=dev)
    ws = torch.empty(A.aps_sync_workspace_bytes(n, L), dtype=torch.uint8, device=dev)
    aps = mode == "aps"
    route = A.aps_sync_route(W, n, pal) if aps else None
    one = route == A.APS_SYNC_ROUTE_ONE_PASS
    guess = route == A.APS_SYNC_ROUTE_GUESS
    ev = []

    def step(record: bool):
        if record:
            e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            e[0].record()
        if aps:
            A.aps_sync(G, n, offs_t, pal, idx_t, A.APS_SYNC_PASS1, mab, se, out, ws)
        if record:
            e[1].record()
        if aps:
            A.aps_sync(G, n, offs_t, pal, idx_t, A.APS_SYNC_PASS2, mab, se, out, ws)
        else:  # casting without APS: no maxima, no scales
            A.aps_sim_reduce(G, n, offs_t, None, pal, idx_t, 0, out=out)
        if record:
            e[2].record()
            ev.append(e)

    for _ in range(warmup):
        step(False)
    torch.cuda.synchronize()
    # the step time: `steps` steps back to back with nothing between them
    runs = []
    for _ in range(loops):
        t0 = time.perf_counter()
        for _ in range(steps):
            step(False)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        runs.append((t1 - t0) * 1e3 / steps)
    ms_per_step = sorted(runs)[len(runs) // 2]
    ms_runs = runs if loops > 1 else None
    # the pass spans: as many steps again, with events around each pass
    for _ in range(steps):
        step(True)
    torch.cuda.synchronize()
    p1 = sum(e[0].elapsed_time(e[1]) for e in ev) / len(ev)
    p2 = sum(e[1].elapsed_time(e[2]) for e in ev) / len(ev)
    assert bool(torch.isfinite(out).all()) or not aps

    graph_ms = None
    if graph:
        # the same step captured once in a HIP graph and replayed: the launches
        # of a step on a set that fits the caches cost more than its work
        eager = out.clone()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step(False)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            step(False)
        for k in range(2):  # replays equal the eager step, before and after the timing
            out.fill_(float("nan"))
            gr.replay()
            torch.cuda.synchronize()
            if not torch.equal(out.view(torch.int32), eager.view(torch.int32)):
                raise RuntimeError("a replay of the captured step differs from the eager step")
            if k == 0:
                for _ in range(warmup):
                    gr.replay()
                torch.cuda.synchronize()
                tg = time.perf_counter()
                for _ in range(steps):
                    gr.replay()
                torch.cuda.synchronize()
                graph_ms = (time.perf_counter() - tg) * 1e3 / steps
        del gr, eager

    rerun = None
    if guess:
        # the layers pass 2 reran: threshold 1 in the workspace's int32[L] part
        up = lambda b: (b + 255) // 256 * 256
        C = (n + 1023) // 1024
        t0_ = up(1024 * C) + up(4 * C)
        rr = ws[t0_:t0_ + 4 * L].cpu().numpy().view("int32") != 0
        rerun = {"layers": int(rr.sum()), "elements": int(sum(sz for sz, r in zip(gs.sizes, rr) if r))}

    # the dominant kernel: the one that reads the W rows and writes the sum
    alg_bytes = 4.0 * W * n + 4.0 * n     # read every worker row once, write the fp32 sum
    if one:
        kernel, k_ms = "k_sync_spec", p1
        note = "pass-1 span: k_sync_spec plus the zeroing of the L maxima (k_sync_clear, a few us)"
        if W >= 128 and all(f.m <= 7 for f in pal):
            # pass 1 keeps each sum in 2 bytes; pass 2 widens them into the fp32 output
            alg_bytes = 4.0 * W * n + 2.0 * n
            note += "; the sums written as 2-byte top halves (pass 2 widens them)"
    elif guess:
        # pass 1 also reads every 32nd worker row for the sampled maxima
        alg_bytes += 4.0 * ((W + 31) // 32) * n
        kernel, k_ms = "k_guess_spec", p1
        note = ("pass-1 span: k_guess_spec plus the sampled maxima (k_maxabs over every 32nd worker row), "
                "bytes of both")
    else:
        kernel, k_ms = "k_sim_reduce", p2
        note = "pass-2 span: k_sim_reduce plus k_scales (a few us)" if aps else "k_sim_reduce alone"
    achieved = alg_bytes / (k_ms * 1e-3) / 1e9
    return {"ms_per_step": ms_per_step, "pass1_ms": p1, "pass2_ms": p2, "aps": aps, "one": one, "guess": guess,
            "route": ("one pass" if one else ("guessed scales" if guess else "two passes")) if aps else "raw reduce",
            "kernel": kernel, "kernel_ms": k_ms, "alg_bytes": alg_bytes, "achieved": achieved, "note": note,
            "rerun": rerun, "graph_ms_per_step": graph_ms, "ms_per_step_runs": ms_runs, "arrays": (mab, se, out, ws)}


# The other workloads timed after the headline step (each also in RAW mode,
# casting without APS): config, palette, and whether its W rows fit the
# 256 MB Infinity Cache (then a step is a few launches, bound by latency).
OTHER_CONFIGS = [("resnet50_w256", "1-4-3", False), ("resnet50_w8", "1-5-2", False),
                 ("bert_large", "hybrid", False), ("resnet20", "1-5-2", True), ("resnet20", "1-4-3", True),
                 ("resnet20", "1-3-0", True), ("mlp", "1-4-3", True)]


def other_configs(A, WL, dev, cfg0: str, pal0: str, held: dict, steps: int, warmup: int) -> dict:
    """Each workload of OTHER_CONFIGS in APS and RAW mode, plus the headline
    set in RAW mode.  held = {"config": cfg0, "gs": the headline GradSet}
    is the only reference to the set in use: the headline set serves its own
    config and is dropped before the next set is drawn."""
    import torch

    res = {}
    plan = [(cfg0, pal0, "raw", False)] + [(c, p, m, cr) for c, p, cr in OTHER_CONFIGS for m in ("aps", "raw")
                                            if (c, p) != (cfg0, pal0)]
    plan.sort(key=lambda x: x[0] != cfg0)  # the headline set's own runs first, while it is held
    for cfg, palette, mode, cache in plan:
        if held["config"] != cfg:
            held["config"], held["gs"] = None, None
            torch.cuda.empty_cache()
            held["gs"] = WL.generate(cfg, palette, device=dev)
            held["config"] = cfg
            torch.cuda.synchronize()
        gs = held["gs"]
        pal = [A.Format(p.e, p.m, p.bias) for p in WL.CONFIGS[cfg].palettes[palette]]
        offs_t = torch.from_numpy(gs.offsets).to(dev)
        idx_t = None if gs.fmt_idx is None else torch.from_numpy(gs.fmt_idx).to(dev)
        m = measure_step(A, gs, pal, idx_t, offs_t, mode, steps, warmup, graph=True, loops=3)
        del m["arrays"]
        W, n = gs.W, gs.n
        res[f"{cfg} {palette} {mode}"] = {
            "W": W, "n": n, "ms_per_step": m["ms_per_step"], "ms_per_step_runs": m["ms_per_step_runs"],
            "elements_per_s": W * n / (m["ms_per_step"] * 1e-3),
            "route": m["route"], "kernel": m["kernel"], "kernel_ms": m["kernel_ms"],
            "algorithmic_bytes_per_launch": m["alg_bytes"], "achieved_GBps": m["achieved"],
            "frac": m["achieved"] / HBM_PEAK_GBPS, "pass1_ms": m["pass1_ms"], "pass2_ms": m["pass2_ms"],
            **({"guess_reruns": m["rerun"]} if m["rerun"] else {}),
            "graph_ms_per_step": m["graph_ms_per_step"],
            "graph_elements_per_s": W * n / (m["graph_ms_per_step"] * 1e-3),
            "residency": ("cache-resident (the W rows fit the 256 MB Infinity Cache; a step is a few launches, "
                          "bound by their latency)") if cache else "HBM",
        }
        print(f"# {cfg} {palette} {mode}: {m['ms_per_step']:.4f} ms/step ({m['graph_ms_per_step']:.4f} as a graph), "
              f"{m['route']}, {m['kernel']} {m['achieved'] / 1e3:.2f} TB/s", file=sys.stderr, flush=True)
        del gs
    held["config"], held["gs"] = None, None
    torch.cuda.empty_cache()
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the multi-GPU path is a design only; this library runs on one GPU)", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration > 0:
        copy_calibration(args.copy_calibration)
        return
    if args.ceilings:
        print(json.dumps(ceilings(args.probe)), flush=True)
        return
    if args.roundoff:
        print(json.dumps({"study": ROUNDOFF_STUDY, "error": roundoff_study()}), flush=True)
        return
    if args.gemm:
        import torch

        from paper_1911_08907_amd import aps as A
        A.lib()
        print(json.dumps(lp_gemm_calls(A, torch.device("cuda:0"))), flush=True)
        return

    import torch

    from paper_1911_08907_amd import aps as A
    from paper_1911_08907_amd import workloads as WL

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    A.lib()
    dev = torch.device("cuda:0")
    cfg = WL.CONFIGS[args.config]
    palette = args.palette or next(iter(cfg.palettes))
    t_gen = time.time()
    gs = WL.generate(args.config, palette, device=dev)
    torch.cuda.synchronize()
    t_gen = time.time() - t_gen
    print(f"# generated {args.config} W={gs.W} n={gs.n} ld={gs.ld} in {t_gen:.1f}s", file=sys.stderr, flush=True)
    pal = [A.Format(p.e, p.m, p.bias) for p in gs.palette]
    W, n, L = gs.W, gs.n, len(gs.sizes)
    offs_t = torch.from_numpy(gs.offsets).to(dev)
    idx_t = None if gs.fmt_idx is None else torch.from_numpy(gs.fmt_idx).to(dev)
    G = gs.G
    aps = args.mode == "aps"
    m = measure_step(A, gs, pal, idx_t, offs_t, args.mode, args.steps, args.warmup, graph=True)
    mab, se, out, _ = m.pop("arrays")
    ms_per_step = m["ms_per_step"]

    other = {}
    if aps:
        other["two_pass_step"] = two_pass_step(A, G, gs, pal, idx_t, offs_t, mab, se, out)
    if not args.no_other_calls:
        other.update(other_calls(A, G, gs, pal, idx_t, offs_t, se if aps else None, out))
        other["lp_gemm"] = lp_gemm_calls(A, dev)

    kernel = m["kernel"]
    traffic, traffic_src = traffic_from_profile(kernel[2:], args.config, palette)
    res = {
        "metric": METRIC,
        "value": W * n / (ms_per_step * 1e-3),
        "unit": "elements/s",
        "reduced_elements_per_s": n / (ms_per_step * 1e-3),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.config, "W": W, "n": n, "tensors": L, "format": palette,
                   "mode": args.mode, "route": m["route"],
                   "layout": "[W][ld] fp32 worker-major, HBM resident"},
        "roofline": {
            "bound": "hbm",
            "achieved": m["achieved"],
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": m["achieved"] / HBM_PEAK_GBPS,
            "traffic": traffic,
            "kernel": kernel,
            "algorithmic_bytes_per_launch": m["alg_bytes"],
            "avg_launch_ms": m["kernel_ms"],
            "timed_span": m["note"],
            "traffic_source": traffic_src,
        },
        "passes_ms": {"pass1": m["pass1_ms"], "pass2": m["pass2_ms"]},
        # the same step captured once in a HIP graph and replayed `steps` times
        # (timed after the eager steps; the replays equal the eager result)
        "graph_ms_per_step": m["graph_ms_per_step"],
        **({"guess_reruns": m["rerun"]} if m["rerun"] else {}),
        "other_calls": other,
        "kernel_source": source_digest(),
    }
    if not args.no_cpu_baseline and aps:
        res["cpu_baseline"] = cpu_baseline(G, gs, pal, args.cpu_seconds)
    if not args.no_other_calls:
        res["roundoff_eq5"] = {"study": ROUNDOFF_STUDY, "error": roundoff_study()}
    held = {"config": args.config, "gs": gs}
    del mab, se, out, G, gs
    if not args.no_other_configs:
        res["other_configs"] = other_configs(A, WL, dev, args.config, palette, held, args.other_steps, 3)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
