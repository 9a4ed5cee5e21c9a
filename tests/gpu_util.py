"""Helpers shared by the GPU tests: run the HIP path on a workload and compare
with the oracle.  Importing this module does not touch the GPU."""
from __future__ import annotations

import numpy as np

import oracle
from tests.invariants import canonical


def device_arrays(wl, device="cuda"):
    import torch

    return (torch.from_numpy(wl.scores).to(device), torch.from_numpy(wl.row_offsets).to(device),
            torch.from_numpy(wl.row_lengths).to(device))


def run_hip(scores, offs, lens, K, policy=None, trace=True, ws=None):
    """One call through the C-ABI.  Returns numpy (idx, val, trace, stats)."""
    import torch
    from paper_2609_08450_amd import topk

    n = int(lens.numel())
    if ws is None:
        ws = topk.alloc_workspace(max(n, 1), K)
    idx = torch.full((n, K), -7, dtype=torch.int32, device=scores.device)
    val = torch.full((n, K), 7.0, dtype=torch.float32, device=scores.device)
    tr = torch.full((n, topk.TRACE_WORDS), -7, dtype=torch.int32, device=scores.device) if trace else None
    topk.read_stats(ws)  # reset counters
    topk.topk_ragged_ex(scores, offs, lens, n, K, idx, val, ws, policy, tr)
    torch.cuda.synchronize()
    st = topk.read_stats(ws)
    return (idx.cpu().numpy(), val.cpu().numpy(), tr.cpu().numpy() if trace else None, st)


def oracle_policy_of(p, K):
    """Oracle policy equal to a library policy (s = 2^s_log2; a negative
    sampling floor -m means m * K)."""
    lmin = p.l_samp_min if p.l_samp_min >= 0 else min(2**31 - 1, -p.l_samp_min * K)
    return oracle.default_policy(s=1 << p.s_log2, rho_num=p.rho_num, rho_den=p.rho_den,
                                 rho1_num=p.rho1_num, rho1_den=p.rho1_den,
                                 l_samp_min=lmin, cap=p.cap)


def assert_same_selection(gi, gv, oi, ov, rows=None, where=""):
    """Per row, the (index, value-bits) sets must be identical."""
    ci, cv = canonical(gi, gv)
    ei, ev = canonical(oi, ov)
    bad = np.nonzero(~(np.all(ci == ei, axis=1) & np.all(cv == ev, axis=1)))[0]
    if bad.size:
        r = int(bad[0])
        rr = rows[r] if rows is not None else r
        d = np.nonzero((ci[r] != ei[r]) | (cv[r] != ev[r]))[0]
        raise AssertionError(f"{where}: {bad.size} rows differ; first row {rr}: "
                             f"{d.size} slots differ, e.g. gpu {ci[r][d[:4]]} vs oracle {ei[r][d[:4]]}")
