"""The allocation-free entry point (topk_ragged_noalloc) against the entry
point with a workspace (topk_ragged), through the C-ABI: identical (index,
value) sets on consecutive calls of shrinking and growing size on the same
device array."""
import numpy as np
import pytest

from paper_2609_08450_amd import workloads as W
from tests.gpu_util import assert_same_selection, device_arrays

pytestmark = pytest.mark.gpu


def _both(topk, wl):
    import torch

    print("[case] noalloc", wl.name, "rows", wl.n_rows, "K", wl.K, flush=True)
    s, o, l = device_arrays(wl)
    n, K = wl.n_rows, wl.K
    ref_i = torch.full((n, K), -7, dtype=torch.int32, device="cuda")
    ref_v = torch.full((n, K), 7.0, dtype=torch.float32, device="cuda")
    ws = topk.alloc_workspace(n, K)
    topk.topk_ragged(s, o, l, n, K, ref_i, ref_v, ws)
    got_i = torch.full((n, K), -9, dtype=torch.int32, device="cuda")
    got_v = torch.full((n, K), 9.0, dtype=torch.float32, device="cuda")
    topk.topk_ragged_noalloc(s, o, l, n, K, got_i, got_v)
    torch.cuda.synchronize()
    assert_same_selection(got_i.cpu().numpy(), got_v.cpu().numpy(), ref_i.cpu().numpy(),
                          ref_v.cpu().numpy(), where=f"noalloc {wl.name}")


def test_noalloc_matches_topk_ragged():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2609_08450_amd import topk

    # two calls in a row, the second smaller (split plans)
    _both(topk, W.decode())
    _both(topk, W.decode(seed=11, n_rows=12))
    # a call of more rows than split rows (one workgroup per row, order
    # pre-pass), then a small one again, then rows at most K and K = 256
    _both(topk, W.adversarial(n_rows=200))
    _both(topk, W.decode(seed=12, n_rows=5))
    _both(topk, W.tiny())


def test_noalloc_mixed_calls_in_a_row():
    """Seeded mixed calls (every row kind, 40 to 1200 rows, K from 256 to
    4096) one after another through the allocation-free entry point, each
    against the oracle: the state the kernels leave in the shared array
    serves the next call whatever its size."""
    import torch

    import oracle
    from paper_2609_08450_amd import topk
    from tests.test_gpu_mixed import mixed_workload

    for seed in range(6):
        wl = mixed_workload(seed)
        n, K = wl.n_rows, wl.K
        print("[case] noalloc mixed seed", seed, "rows", n, "K", K, flush=True)
        s, o, l = device_arrays(wl)
        gi = torch.full((n, K), -9, dtype=torch.int32, device="cuda")
        gv = torch.full((n, K), 9.0, dtype=torch.float32, device="cuda")
        topk.topk_ragged_noalloc(s, o, l, n, K, gi, gv)
        torch.cuda.synchronize()
        oi, ov = oracle.topk_ragged(wl.scores, wl.row_offsets, wl.row_lengths, K)
        assert_same_selection(gi.cpu().numpy(), gv.cpu().numpy(), oi, ov,
                              where=f"noalloc mixed seed {seed}")


def test_noalloc_rejects_too_many_rows():
    import torch

    from paper_2609_08450_amd import topk

    n = 16385
    e = torch.zeros(1, device="cuda")
    with pytest.raises(topk.TopkError, match="workspace too small"):
        topk.topk_ragged_noalloc(e, torch.zeros(n, dtype=torch.int64, device="cuda"),
                                 torch.zeros(n, dtype=torch.int32, device="cuda"), n, 2048,
                                 torch.empty((n, 2048), dtype=torch.int32, device="cuda"),
                                 torch.empty((n, 2048), dtype=torch.float32, device="cuda"))
