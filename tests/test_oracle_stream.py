"""The streamed oracle (row blocks for the maxima, column slices for the
sum) equals one oracle call over the whole set (CPU only).  The full-size
GPU parity tests rely on it."""
import numpy as np
import pytest

import oracle as O
from tests._util import first_diff, same_f32
from tests.oracle_stream import oracle_maxabs, oracle_sum_sliced


@pytest.mark.parametrize("cols", [1, 7, 64, 1000])
def test_streamed_oracle_equals_one_call(cols):
    rng = np.random.default_rng(5)
    sizes = [0, 3, 63, 2, 0, 69, 1, 700, 0]
    offs = np.zeros(len(sizes) + 1, np.int64)
    offs[1:] = np.cumsum(sizes)
    n = int(offs[-1])
    W = 5
    host = (rng.standard_normal((W, n)) * np.repeat(10.0 ** rng.uniform(-8, 0, len(sizes)), sizes)).astype(np.float32)
    host[1, 5] = np.inf
    host[3, 80] = np.nan
    opal = [O.Format(5, 10), O.Format(5, 2)]
    fi = (np.arange(len(sizes)) % 2).astype(np.uint8)
    mab = oracle_maxabs(host, n, offs)
    assert np.array_equal(mab, O.layer_maxabs(host, n, offs))
    se = O.layer_scales(mab, W, opal, fi)
    for s in (se, None):
        a = oracle_sum_sliced(host, n, offs, s, opal, fi, "slicing", cols=cols)
        b = O.sim_reduce(host, n, offs, s, opal, fi)
        assert same_f32(a, b), first_diff(a, b)
