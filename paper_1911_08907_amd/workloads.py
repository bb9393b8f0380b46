"""Seeded synthetic gradient sets shaped like the paper's models.

This module only draws inputs: it holds none of the APS arithmetic.  Both the
HIP path (tests, benchmark) and the CPU oracle consume what it produces.

A gradient set is W workers' flat fp32 gradients stored worker-major as a
[W][ld] tensor (ld = n rounded up to 256, zero padded: rows of fp32 start on
1 KB boundaries and rows of 8-bit codes with the same stride on 256-byte
ones, so no row shares a cache line with the next), plus the int64 layer
offsets (one layer per parameter tensor, in parameter-registration order),
and a per-layer palette index.

Value recipe (per tensor i, shared by all workers: a scale s_i drawn
log-uniformly in [lo, hi]; per worker and element):
  * values ~ Normal(0, s_i^2);
  * each element independently set to +0 with probability ``zero_p``;
  * each element independently replaced, with probability ``outlier_p``, by
    outlier_scale * s_i * T, T ~ Student-t(2) = Z / sqrt(-ln U);
  * for tensors listed in ``sparse_rows``: each row (last-dim slice) is all
    zero with probability ``sparse_p``, independently per worker.
Random draws: numpy PCG64 for the per-tensor scales (seed = (base, config,
"scales")); torch's generator on the target device for the values, one
generator per worker seeded from (base, config, worker).  Values therefore
depend on the device type; parity tests always hand the oracle the exact
bytes the GPU consumed.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field
from typing import Callable

import numpy as np

BASE_SEED = 1911


# ----------------------------------------------------------------- shapes

def mlp_shapes():
    """784-128-10 MLP: fc1 weight/bias, fc2 weight/bias."""
    return [("fc1.weight", (128, 784)), ("fc1.bias", (128,)),
            ("fc2.weight", (10, 128)), ("fc2.bias", (10,))]


def _bn(prefix, c):
    return [(f"{prefix}.weight", (c,)), (f"{prefix}.bias", (c,))]


def resnet20_shapes():
    """CIFAR ResNet-20 (3 stages x 3 basic blocks, widths 16/32/64) with 1x1
    projection shortcuts where the width or stride changes; 64x10 FC."""
    s = [("conv1.weight", (16, 3, 3, 3))] + _bn("bn1", 16)
    cin = 16
    for st, w in enumerate((16, 32, 64)):
        for b in range(3):
            p = f"layer{st + 1}.{b}"
            s.append((f"{p}.conv1.weight", (w, cin, 3, 3)))
            s += _bn(f"{p}.bn1", w)
            s.append((f"{p}.conv2.weight", (w, w, 3, 3)))
            s += _bn(f"{p}.bn2", w)
            if b == 0 and cin != w:
                s.append((f"{p}.shortcut.0.weight", (w, cin, 1, 1)))
                s += _bn(f"{p}.shortcut.1", w)
            cin = w
    s += [("fc.weight", (10, 64)), ("fc.bias", (10,))]
    return s


def resnet50_shapes():
    """ImageNet ResNet-50 (bottlenecks 3/4/6/3, expansion 4, downsample on the
    first block of each stage), 2048x1000 FC."""
    s = [("conv1.weight", (64, 3, 7, 7))] + _bn("bn1", 64)
    cin = 64
    for st, (w, nb) in enumerate(zip((64, 128, 256, 512), (3, 4, 6, 3))):
        for b in range(nb):
            p = f"layer{st + 1}.{b}"
            s.append((f"{p}.conv1.weight", (w, cin, 1, 1)))
            s += _bn(f"{p}.bn1", w)
            s.append((f"{p}.conv2.weight", (w, w, 3, 3)))
            s += _bn(f"{p}.bn2", w)
            s.append((f"{p}.conv3.weight", (4 * w, w, 1, 1)))
            s += _bn(f"{p}.bn3", 4 * w)
            if b == 0:
                s.append((f"{p}.downsample.0.weight", (4 * w, cin, 1, 1)))
                s += _bn(f"{p}.downsample.1", 4 * w)
            cin = 4 * w
    s += [("fc.weight", (1000, 2048)), ("fc.bias", (1000,))]
    return s


def bert_large_shapes():
    """BERT-large (24 layers, hidden 1024, FFN 4096, vocab 30522, 512
    positions, 2 token types) with the pooler."""
    H, F = 1024, 4096
    s = [("embeddings.word_embeddings.weight", (30522, H)),
         ("embeddings.position_embeddings.weight", (512, H)),
         ("embeddings.token_type_embeddings.weight", (2, H)),
         ("embeddings.LayerNorm.weight", (H,)), ("embeddings.LayerNorm.bias", (H,))]
    for i in range(24):
        p = f"encoder.layer.{i}"
        for nm in ("query", "key", "value"):
            s += [(f"{p}.attention.self.{nm}.weight", (H, H)), (f"{p}.attention.self.{nm}.bias", (H,))]
        s += [(f"{p}.attention.output.dense.weight", (H, H)), (f"{p}.attention.output.dense.bias", (H,)),
              (f"{p}.attention.output.LayerNorm.weight", (H,)), (f"{p}.attention.output.LayerNorm.bias", (H,)),
              (f"{p}.intermediate.dense.weight", (F, H)), (f"{p}.intermediate.dense.bias", (F,)),
              (f"{p}.output.dense.weight", (H, F)), (f"{p}.output.dense.bias", (H,)),
              (f"{p}.output.LayerNorm.weight", (H,)), (f"{p}.output.LayerNorm.bias", (H,))]
    s += [("pooler.dense.weight", (H, H)), ("pooler.dense.bias", (H,))]
    return s


# ---------------------------------------------------------------- configs

@dataclass(frozen=True)
class FormatSpec:
    e: int
    m: int
    bias: int | None = None


@dataclass
class Config:
    name: str
    shapes: Callable
    W: int
    palettes: dict            # palette name -> list of FormatSpec
    scale_lo: float
    scale_hi: float
    zero_p: float = 0.0
    outlier_p: float = 0.0
    outlier_scale: float = 100.0
    sparse_rows: tuple = ()   # tensor names whose rows are zeroed
    sparse_p: float = 0.0
    palette_of: Callable | None = None   # tensor name -> palette index
    cid: int = 0


E5M2, E4M3, E3M0, E5M10 = FormatSpec(5, 2), FormatSpec(4, 3), FormatSpec(3, 0), FormatSpec(5, 10)


def _bert_palette(name: str) -> int:
    # word, position and token-type embeddings at 1-5-10, everything else 1-5-2
    return 0 if name.endswith("_embeddings.weight") else 1


CONFIGS = {
    "mlp": Config("mlp", mlp_shapes, 2, {"1-4-3": [E4M3]}, 1e-5, 1e-1, zero_p=0.01, cid=1),
    "resnet20": Config("resnet20", resnet20_shapes, 8,
                       {"1-5-2": [E5M2], "1-4-3": [E4M3], "1-3-0": [E3M0]}, 1e-6, 1e-1,
                       outlier_p=1e-4, outlier_scale=100.0, cid=2),
    "resnet50_w8": Config("resnet50_w8", resnet50_shapes, 8, {"1-5-2": [E5M2]}, 1e-7, 1e-1,
                          zero_p=0.02, cid=3),
    "resnet50_w256": Config("resnet50_w256", resnet50_shapes, 256, {"1-5-2": [E5M2], "1-4-3": [E4M3]},
                            1e-7, 1e-1, zero_p=0.02, cid=4),
    "bert_large": Config("bert_large", bert_large_shapes, 8, {"hybrid": [E5M10, E5M2]}, 1e-7, 1e-2,
                         sparse_rows=("embeddings.word_embeddings.weight",
                                      "embeddings.position_embeddings.weight"),
                         sparse_p=0.95, palette_of=_bert_palette, cid=5),
}


def _seed(*parts) -> int:
    h = hashlib.sha256(repr(parts).encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


@dataclass
class GradSet:
    config: str
    W: int
    n: int
    ld: int
    names: list
    sizes: list
    offsets: np.ndarray          # int64[L+1]
    palette: list                # FormatSpec list
    fmt_idx: np.ndarray | None   # uint8[L] or None
    G: object = None             # torch tensor [W][ld] float32
    scales: np.ndarray = field(default=None)


def layout(cfg_name: str):
    cfg = CONFIGS[cfg_name]
    shapes = cfg.shapes()
    names = [nm for nm, _ in shapes]
    sizes = [int(np.prod(sh)) for _, sh in shapes]
    offs = np.zeros(len(sizes) + 1, np.int64)
    offs[1:] = np.cumsum(sizes)
    return cfg, shapes, names, sizes, offs


def generate(cfg_name: str, palette: str | None = None, device="cpu", seed: int = BASE_SEED,
             W: int | None = None) -> GradSet:
    """Draw the gradient set of a config on ``device`` (a torch device)."""
    import torch

    cfg, shapes, names, sizes, offs = layout(cfg_name)
    W = cfg.W if W is None else W
    n = int(offs[-1])
    ld = (n + 255) // 256 * 256
    pal_name = palette or next(iter(cfg.palettes))
    pal = cfg.palettes[pal_name]
    fmt_idx = None
    if cfg.palette_of is not None:
        fmt_idx = np.array([cfg.palette_of(nm) for nm in names], np.uint8)

    rs = np.random.Generator(np.random.PCG64(_seed(seed, cfg.cid, "scales")))
    s = np.exp(rs.uniform(np.log(cfg.scale_lo), np.log(cfg.scale_hi), len(sizes))).astype(np.float32)

    dev = torch.device(device)
    scale_vec = torch.from_numpy(np.repeat(s, sizes)).to(dev)
    G = torch.zeros((W, ld), dtype=torch.float32, device=dev)
    row_groups = []
    for nm in cfg.sparse_rows:
        i = names.index(nm)
        rows, cols = shapes[i][1][0], int(np.prod(shapes[i][1][1:]))
        row_groups.append((int(offs[i]), rows, cols))
    g = torch.Generator(device=dev)
    for w in range(W):
        g.manual_seed(_seed(seed, cfg.cid, "worker", w))
        row = G[w, :n]
        torch.randn(n, generator=g, device=dev, out=row)
        row.mul_(scale_vec)
        if cfg.zero_p > 0:
            row.masked_fill_(torch.rand(n, generator=g, device=dev) < cfg.zero_p, 0.0)
        if cfg.outlier_p > 0:
            mask = torch.rand(n, generator=g, device=dev) < cfg.outlier_p
            k = int(mask.sum())
            if k:
                z = torch.randn(k, generator=g, device=dev)
                u = torch.rand(k, generator=g, device=dev).clamp_min(1e-30)
                t = z / torch.sqrt(-torch.log(u))
                row[mask] = (cfg.outlier_scale * scale_vec[mask] * t).to(torch.float32)
        for start, rows, cols in row_groups:
            zr = torch.rand(rows, generator=g, device=dev) < cfg.sparse_p
            row[start:start + rows * cols].view(rows, cols).masked_fill_(zr[:, None], 0.0)
    return GradSet(cfg_name, W, n, ld, names, sizes, offs, list(pal), fmt_idx, G, s)
