"""The oracle over sets too large for one call of a few seconds (test
infrastructure; no APS arithmetic of its own).

The layer maxima are taken on blocks of worker rows in parallel threads (the
oracle's maximum is a maximum of bit patterns, so grouping the rows does not
change it), and the rounded W-worker sum on successive column slices of all
W rows, each slice with the full layers' exponents."""
from __future__ import annotations

import os
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle as O
from tests._util import log

SLICE = 1 << 17       # columns per oracle call (all W rows)
THREADS = max(1, min(16, os.cpu_count() or 1))


def oracle_maxabs(host, n, offsets):
    """The oracle's per-layer maxima over all rows, row blocks in parallel."""
    W = host.shape[0]
    blocks = [b for b in np.array_split(np.arange(W), min(W, THREADS)) if b.size]

    def part(rows):
        return O.layer_maxabs(host[rows[0]:rows[-1] + 1], n, offsets).view(np.uint32)

    with ThreadPoolExecutor(len(blocks)) as ex:
        parts = list(ex.map(part, blocks))
    return np.maximum.reduce(parts)


def oracle_sum_sliced(host, n, offsets, scale_exp, opal, fmt_idx, tag, cols=SLICE):
    """The oracle's rounded W-worker sum over successive column slices."""
    out = np.empty(n, np.float32)
    t0, last = time.time(), time.time()
    for c0 in range(0, n, cols):
        c1 = min(n, c0 + cols)
        i0 = int(np.searchsorted(offsets, c0, side="right")) - 1
        i1 = int(np.searchsorted(offsets, c1 - 1, side="right")) - 1
        sub = (np.clip(offsets[i0:i1 + 2], c0, c1) - c0).astype(np.int64)
        se = None if scale_exp is None else scale_exp[i0:i1 + 1]
        fi = None if fmt_idx is None else fmt_idx[i0:i1 + 1]
        block = np.ascontiguousarray(host[:, c0:c1])
        out[c0:c1] = O.sim_reduce(block, c1 - c0, sub, se, opal, fi)
        if time.time() - last > 20:
            last = time.time()
            log(f"  {tag}: oracle at column {c1} of {n}, {last - t0:.0f}s")
    log(f"  {tag}: oracle sum of {host.shape[0]} x {n} in {time.time() - t0:.1f}s")
    return out
