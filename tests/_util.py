"""Helpers shared by the tests (no APS arithmetic here)."""
from __future__ import annotations

import sys

import numpy as np

import oracle as O


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def ofmt(f) -> O.Format:
    """Binding/workload format -> oracle format (same numbers, separate type)."""
    return O.Format(f.e, f.m, getattr(f, "bias", None))


def same_f32(a, b) -> bool:
    """Bitwise equality of float32 arrays, any NaN equal to any NaN."""
    a = np.ascontiguousarray(a, np.float32)
    b = np.ascontiguousarray(b, np.float32)
    if a.shape != b.shape:
        return False
    na, nb = np.isnan(a), np.isnan(b)
    if not np.array_equal(na, nb):
        return False
    return np.array_equal(a.view(np.uint32)[~na], b.view(np.uint32)[~nb])


def first_diff(a, b, k=5):
    a = np.ascontiguousarray(a, np.float32).ravel()
    b = np.ascontiguousarray(b, np.float32).ravel()
    na, nb = np.isnan(a), np.isnan(b)
    bad = (na != nb) | (~na & ~nb & (a.view(np.uint32) != b.view(np.uint32)))
    idx = np.nonzero(bad)[0][:k]
    return [(int(i), float(a[i]), float(b[i])) for i in idx], int(bad.sum())


def same_maxabs(a, b) -> bool:
    a = np.asarray(a).view(np.uint32)
    b = np.asarray(b).view(np.uint32)
    an, bn = a > 0x7F800000, b > 0x7F800000
    return np.array_equal(an, bn) and np.array_equal(a[~an], b[~bn])
