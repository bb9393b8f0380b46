"""The binding's refusals on GPU tensors: wrong dtypes, too few elements,
non-contiguous arrays, a G narrower than n, Q with another row stride than
X, a GEMM output of the wrong shape.  Each is a ValueError raised before the
library is called; a correct call right after still equals the oracle."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_1911_08907_amd import aps as A
from tests._util import ofmt, same_f32

pytestmark = pytest.mark.gpu

F = A.Format


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    A.lib()
    return torch.device("cuda:0")


def test_bad_arrays_are_refused(dev):
    W, n, ld = 3, 1000, 1024
    G = torch.randn(W, ld, device=dev) * 1e-3
    offs = torch.tensor([0, 400, 1000], dtype=torch.int64, device=dev)
    i32 = lambda k: torch.zeros(k, dtype=torch.int32, device=dev)  # noqa: E731
    bad = {
        "G float64": lambda: A.aps_sync(G.double(), n, offs, [F(5, 2)]),
        "G narrower than n": lambda: A.aps_sync(G[:, :900], n, offs, [F(5, 2)]),
        "G transposed": lambda: A.aps_layer_maxabs(G.t().contiguous().t(), n, offs, i32(2)),
        "offsets int32": lambda: A.aps_sync(G, n, offs.int(), [F(5, 2)]),
        "maxabs_bits too short": lambda: A.aps_layer_maxabs(G, n, offs, i32(1)),
        "scale_exp float": lambda: A.aps_layer_scales(i32(2), W, [F(5, 2)], None, torch.zeros(2, device=dev)),
        "fmt_idx int64": lambda: A.aps_sim_reduce(G, n, offs, None, [F(5, 2), F(4, 3)],
                                                  torch.zeros(2, dtype=torch.int64, device=dev), 0,
                                                  out=torch.zeros(n, device=dev)),
        "out too short": lambda: A.aps_sim_reduce(G, n, offs, None, [F(5, 2)], None, 0,
                                                  out=torch.zeros(n - 1, device=dev)),
        "out non-contiguous": lambda: A.aps_sim_reduce(G, n, offs, None, [F(5, 2)], None, 0,
                                                       out=torch.zeros(2 * n, device=dev)[::2]),
        "codes too short": lambda: A.aps_quantize(G, n, offs, None, [F(5, 2)], None,
                                                  codes=torch.zeros(W * ld - 1, dtype=torch.uint8, device=dev)),
        "Q another row stride": lambda: A.aps_quantize(G, n, offs, None, [F(5, 2)], None,
                                                       Q=torch.zeros(W, ld + 4, device=dev)[:, :ld]),
        "dequantize codes too short": lambda: A.aps_dequantize(None, torch.zeros(n - 1, dtype=torch.uint8, device=dev),
                                                               n, offs, None, [F(5, 2)], None,
                                                               torch.zeros(n, device=dev)),
        "workspace too short for its dtype": lambda: A.aps_sync(G, n, offs, [F(5, 2)],
                                                                workspace=torch.zeros(8, device=dev)),
        "GEMM C shape": lambda: A.aps_lp_gemm(torch.zeros(4, 8, device=dev), torch.zeros(8, 5, device=dev),
                                             F(5, 2), F(5, 10), C=torch.zeros(5, 4, device=dev)),
        "GEMM A int": lambda: A.aps_lp_gemm(torch.zeros(4, 8, dtype=torch.int32, device=dev),
                                           torch.zeros(8, 5, device=dev), F(5, 2), F(5, 10)),
    }
    for name, call in bad.items():
        with pytest.raises(ValueError):
            call()
        torch.cuda.synchronize()
    # the library is untouched by the refusals: a correct call equals the oracle
    out, se, mab, _ = A.aps_sync(G, n, offs, [F(5, 2)])
    torch.cuda.synchronize()
    Gh, oh = G.cpu().numpy(), offs.cpu().numpy()
    o_se = O.layer_scales(O.layer_maxabs(Gh, n, oh), W, [ofmt(F(5, 2))])
    assert np.array_equal(se.cpu().numpy(), o_se)
    assert same_f32(out.cpu().numpy(), O.sim_reduce(Gh, n, oh, o_se, [ofmt(F(5, 2))]))
