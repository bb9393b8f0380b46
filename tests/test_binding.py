"""The Python binding refuses arrays the C ABI could not use (CPU tensors,
wrong dtypes, too few elements, other devices) before anything reaches the
library, so a caller's mistake becomes a ValueError and never a bad device
pointer.  These run without a GPU: CPU tensors are refused first."""
import pytest
import torch

from paper_1911_08907_amd import aps as A

F = A.Format


def _cpu_set():
    G = torch.zeros(2, 8)
    offs = torch.tensor([0, 3, 8], dtype=torch.int64)
    return G, offs


CALLS = {
    "aps_layer_maxabs": lambda G, o: A.aps_layer_maxabs(G, 8, o, torch.zeros(2, dtype=torch.int32)),
    "aps_layer_scales": lambda G, o: A.aps_layer_scales(torch.zeros(2, dtype=torch.int32), 2, [F(5, 2)], None,
                                                        torch.zeros(2, dtype=torch.int32)),
    "aps_quantize": lambda G, o: A.aps_quantize(G, 8, o, None, [F(5, 2)], None, Q=G),
    "aps_sim_reduce": lambda G, o: A.aps_sim_reduce(G, 8, o, None, [F(5, 2)], None, 0, out=torch.zeros(8)),
    "aps_sim_reduce_ex": lambda G, o: A.aps_sim_reduce_ex(G, 8, o, None, [F(5, 2)], None, 0, out=torch.zeros(8)),
    "aps_sim_reduce_codes": lambda G, o: A.aps_sim_reduce_codes(torch.zeros(16, dtype=torch.uint8), 2, 8, 8, o, None,
                                                                [F(5, 2)], None, 0, out=torch.zeros(8)),
    "aps_dequantize": lambda G, o: A.aps_dequantize(None, torch.zeros(8, dtype=torch.uint8), 8, o, None, [F(5, 2)],
                                                    None, torch.zeros(8)),
    "aps_lp_gemm": lambda G, o: A.aps_lp_gemm(torch.zeros(2, 2), torch.zeros(2, 2), F(5, 2), F(5, 10)),
    "aps_sync": lambda G, o: A.aps_sync(G, 8, o, [F(5, 2)]),
    "aps_sync_noalloc": lambda G, o: A.aps_sync_noalloc(G, 8, o, [F(5, 2)], None, torch.zeros(2, dtype=torch.int32),
                                                        torch.zeros(2, dtype=torch.int32), torch.zeros(8)),
    "aps_step": lambda G, o: A.aps_step(G, 8, o, [F(5, 2)]),
}


@pytest.mark.parametrize("name", sorted(CALLS))
def test_cpu_tensors_are_refused(name):
    G, offs = _cpu_set()
    with pytest.raises(ValueError, match="GPU tensor"):
        CALLS[name](G, offs)


def test_every_compute_call_is_covered():
    compute = [nm for nm in A.EXPORTS if nm not in ("aps_format_supported", "aps_sync_workspace_bytes",
                                                     "aps_sync_route", "aps_strerror")]
    assert sorted(compute) == sorted(nm for nm in CALLS if nm != "aps_step")
