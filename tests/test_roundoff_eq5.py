"""The Eq. (5) figure the benchmark reports (bench.round_off_error, numpy)
against the oracle's pinned oracle_round_off_error: on random arrays with
zeros in grad_h on the CPU, and on the very arrays of the group-size study
on the GPU, where the study's low-precision reductions are also checked
against the oracle's hierarchical-order reduce."""
import numpy as np
import pytest

import bench
import oracle as O
from tests._util import first_diff, same_f32


def test_round_off_error_matches_the_oracle():
    rng = np.random.default_rng(55)
    for n in (1, 7, 1000, 65537):
        h = (rng.standard_normal(n) * 10.0 ** rng.uniform(-30, 30, n)).astype(np.float32)
        lo = (h * (1 + rng.standard_normal(n) * 0.3)).astype(np.float32)
        h[rng.random(n) < 0.2] = 0.0
        lo[rng.random(n) < 0.1] = 0.0
        a, b = bench.round_off_error(h, lo), O.round_off_error(h, lo)
        assert a == pytest.approx(b, rel=1e-12, abs=0), (n, a, b)
    # every grad_h zero: no element counts
    z = np.zeros(5, np.float32)
    assert bench.round_off_error(z, np.ones(5, np.float32)) == O.round_off_error(z, np.ones(5, np.float32)) == 0.0
    # a value and its own rounding: 1 -> 0.75 is 25 %, 4 -> 4 is 0
    h = np.array([1.0, 4.0, 0.0], np.float32)
    lo = np.array([0.75, 4.0, 9.0], np.float32)
    assert bench.round_off_error(h, lo) == O.round_off_error(h, lo) == pytest.approx(0.125, abs=0)


@pytest.mark.gpu
def test_roundoff_study_matches_the_oracle():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1911_08907_amd import aps as A

    A.lib()
    n = 64 * 3 * 7 * 7
    offs = np.array([0, n], np.int64)
    for name, (G, se, h, lows) in bench.roundoff_arrays().items():
        # grad_h: the fp32 all-reduce in worker order
        o_h = O.sim_reduce(G, n, offs, None, O.Format(8, 23))
        assert same_f32(h, o_h), (name, first_diff(h, o_h))
        for key, lo in lows.items():
            k = 1 if key == "ring_256" else int(key.split("_")[1])
            o_l = O.sim_reduce_ex(G, n, offs, se, O.Format(5, 2), group=k)
            assert same_f32(lo, o_l), (name, key, first_diff(lo, o_l))
            a, b = bench.round_off_error(h, lo), O.round_off_error(h, lo)
            assert a == pytest.approx(b, rel=1e-12, abs=0), (name, key, a, b)
