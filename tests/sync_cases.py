"""Input generators for the one-pass synchronisation tests (CPU and GPU):
layers whose inputs sit at, around and below the threshold 2^(emin - ft)
below which the unscaled sum may differ from the scaled one.  The layer's
exponent ft comes from the oracle."""
from __future__ import annotations

import numpy as np

import oracle as O


def threshold_values(rng, W, ld, offs, f, layer_max):
    """Each layer i gets its maximum layer_max[i] at worker 0, element 0;
    about a tenth of the other entries sit at, just above or just below the
    layer's threshold 2^(emin - ft), at half, three quarters, 1.5x and 3x of
    it, at the format's half-smallest-subnormal after scaling, or in or at
    the edge of fp32's subnormal range; in a twentieth of the columns worker
    1 cancels worker 0 exactly."""
    L = offs.size - 1
    G = np.zeros((W, ld), np.float32)
    emin = 1 - f.b
    of = O.Format(f.e, f.m, f.bias)
    for i in range(L):
        a, b = offs[i], offs[i + 1]
        if b == a:
            continue
        M = np.float32(layer_max[i])
        ft = O.scale_one(int(M.view(np.uint32)), W, of)
        T = np.float32(2.0 ** (emin - ft)) if -149 <= emin - ft <= 127 else np.float32(0)
        h = emin - ft - f.m - 1
        vals = np.clip((rng.standard_normal((W, b - a)) * M / 4).astype(np.float32), -M, M)
        pick = rng.random((W, b - a)) < 0.1
        with np.errstate(over="ignore"):
            cand = np.array([T, np.nextafter(T, np.float32(1)), np.nextafter(T, np.float32(0)), T / 2, T * 0.75,
                             T * 1.5, T * 3, np.float32(2.0 ** h) if h >= -149 else 0, np.float32(1e-40),
                             np.float32(2.0 ** -126), np.nextafter(np.float32(2.0 ** -126), np.float32(0))],
                            np.float32)
        sgn = np.where(rng.random((W, b - a)) < 0.5, -1, 1).astype(np.float32)
        vals[pick] = cand[rng.integers(0, cand.size, int(pick.sum()))] * sgn[pick]
        if W >= 2:
            cc = rng.random(b - a) < 0.05
            vals[1, cc] = -vals[0, cc]
        vals[0, 0] = M
        G[:, a:b] = vals
    G[:, offs[-1]:] = np.nan
    return G


LAYER_MAXIMA = [1.0, 2.0 ** -100, 3.7e-3, 1e30, 2.0 ** -140, 1.5, 6e37, 1.0 / 3]
