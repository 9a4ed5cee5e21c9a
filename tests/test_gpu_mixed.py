"""Seeded mixed calls: every row kind the selector routes differently, and
special FP32 values, in one call, at random lengths, buffer positions and
alignments, for both kernel instances (calls of at most and of more than
2 x CUs rows) and several K; selections and route traces compared with the
oracle, bit-exact."""
import os

import numpy as np
import pytest

from paper_2609_08450_amd import workloads as W
from tests.test_gpu_parity import parity, say, topk  # noqa: F401  (topk: the fixture)

pytestmark = pytest.mark.gpu

KINDS = ("decode", "codebook", "view low", "view high", "minus inf", "hot block",
         "copies of one", "constant", "specials")

# +-inf, +-0, the largest finite values, the smallest normals, subnormals, and
# values around FP16's largest finite (65504) and smallest subnormal (2^-24)
SPECIALS = np.array([np.inf, -np.inf, 0.0, -0.0, 3.4028235e38, -3.4028235e38,
                     1.1754944e-38, -1.1754944e-38, 1e-45, -1e-45, 3e-39, -3e-39,
                     65504.0, 65520.0, -65520.0, 5.96e-8, 2.98e-8, -2.98e-8], np.float32)


def mixed_row(rng, kind, L, phase):
    """A row of length L of the given kind (phase: the row's view phase at
    stride 128, which the strided kinds target)."""
    if L == 0:
        return np.zeros(0, np.float32)
    x = W.decode_mixture_row(rng, L).astype(np.float32)
    if kind == "codebook":
        book = np.unique(rng.standard_normal(4096).astype(np.float32))[:int(rng.integers(2, 300))]
        x = book[rng.integers(0, book.size, L)]
    elif kind == "view low":
        x[phase::128] = rng.normal(-2.0, 1.0, x[phase::128].size).astype(np.float32)
    elif kind == "view high":
        x[phase::128] = rng.normal(3.0, 0.5, x[phase::128].size).astype(np.float32)
    elif kind == "minus inf":
        x[rng.random(L) < rng.uniform(0.2, 0.999)] = -np.inf
    elif kind == "hot block":
        a = int(rng.integers(0, L))
        b = min(L, a + int(rng.integers(1, 6000)))
        x[a:b] = rng.normal(4.0, 0.1, b - a).astype(np.float32)
    elif kind == "copies of one":
        x = rng.normal(-3.0, 0.5, L).astype(np.float32)
        x[rng.choice(L, min(L, 10000), replace=False)] = 1.0
    elif kind == "constant":
        x[:] = np.float32(rng.choice([0.0, -0.0, 1.5, -np.inf]))
    elif kind == "specials":
        m = rng.random(L) < rng.uniform(0.01, 0.9)
        x[m] = SPECIALS[rng.integers(0, SPECIALS.size, int(m.sum()))]
    return x.astype(np.float32, copy=False)


def mixed_workload(seed):
    rng = np.random.default_rng(9000 + seed)
    n = int(rng.choice([40, 300, 700, 1200]))
    K = int(rng.choice([2048, 2048, 256, 1024, 4096]))
    u = rng.random(n)
    lens = np.floor(np.exp(np.log(1.0) + u * np.log(300000.0))).astype(np.int64) - 1
    lens[rng.random(n) < 0.05] = 0
    lens[rng.random(n) < 0.05] = K
    # a few long rows, so that both the plan and the item table cut some
    longs = rng.choice(n, max(1, n // 40), replace=False)
    lens[longs] = rng.integers(150000, 600000, longs.size)
    lens = np.minimum(lens, 600000)
    parts, offs, pos = [], np.zeros(n, np.int64), 0
    for r in rng.permutation(n):               # buffer order differs from row order
        gap = int(rng.integers(0, 9))           # any 4-byte alignment
        parts.append(np.zeros(gap, np.float32))
        pos += gap
        kind = KINDS[int(rng.integers(0, len(KINDS)))]
        phase = int(format(int(r) % 128, "07b")[::-1], 2)
        x = mixed_row(rng, kind, int(lens[r]), phase)
        parts.append(x)
        offs[r] = pos
        pos += x.size
    buf = np.concatenate(parts + [np.zeros(8, np.float32)])
    return W.Workload(f"mixed seed {seed}", buf, offs, lens.astype(np.int32), K,
                      f"{n} mixed rows, K={K}")


def _seeds():
    """Seeds 0-5, or the range TOPK_MIXED_SEEDS=a:b (a wider sweep)."""
    a, b = os.environ.get("TOPK_MIXED_SEEDS", "0:6").split(":")
    return range(int(a), int(b))


@pytest.mark.parametrize("seed", _seeds())
def test_mixed_call(topk, seed):
    wl = mixed_workload(seed)
    say("mixed", seed, "rows", wl.n_rows, "K", wl.K, "sum L", wl.total_len)
    gt, st = parity(topk, wl, where=f"mixed seed {seed}", per_k=True)
    say("routes", st)
    assert st["errors"] == 0


@pytest.mark.parametrize("seed", range(3))
def test_mixed_call_one_poll(topk, seed):
    """The same calls with one poll allowed for every bounded wait, so that
    segments stop waiting for the boundaries or the route word and take their
    fallbacks (building the view themselves, leaving their range to the last
    arrival): the same selections and traces."""
    wl = mixed_workload(seed)
    topk.debug_set_spin_limit(1)
    try:
        gt, st = parity(topk, wl, where=f"mixed seed {seed}, one poll", per_k=True)
    finally:
        topk.debug_set_spin_limit(0)
    say("routes", st)
    assert st["errors"] == 0


@pytest.mark.parametrize("seed", range(2))
def test_mixed_call_graph_replays(topk, seed):
    """A mixed call captured in a HIP graph and replayed three times, with an
    eager call of another mix on the same workspace between replays: every
    replay and every eager call equal the oracle (the kernels leave the
    workspace's state as they found it, whatever routes a call took)."""
    import torch

    import oracle
    from tests.gpu_util import assert_same_selection, device_arrays

    wl, other = mixed_workload(seed), mixed_workload(seed + 1000)
    n, K, n2, K2 = wl.n_rows, wl.K, other.n_rows, other.K
    say("graph", seed, "rows", n, "K", K, "between", n2, K2)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        s, o, l = device_arrays(wl)
        s2, o2, l2 = device_arrays(other)
        ws = topk.alloc_workspace(max(n, n2), max(K, K2), torch.device("cuda", 0), stream)
        gi = torch.full((n, K), -9, dtype=torch.int32, device="cuda")
        gv = torch.full((n, K), 9.0, dtype=torch.float32, device="cuda")
        ei = torch.empty((n2, K2), dtype=torch.int32, device="cuda")
        ev = torch.empty((n2, K2), dtype=torch.float32, device="cuda")
    stream.synchronize()
    topk.topk_ragged(s, o, l, n, K, gi, gv, ws, stream)
    stream.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        topk.topk_ragged(s, o, l, n, K, gi, gv, ws, torch.cuda.current_stream())
    stream.synchronize()
    oi, ov = oracle.topk_ragged(wl.scores, wl.row_offsets, wl.row_lengths, K)
    oi2, ov2 = oracle.topk_ragged(other.scores, other.row_offsets, other.row_lengths, K2)
    for rep in range(3):
        with torch.cuda.stream(stream):
            gi.fill_(-9)
            gv.fill_(9.0)
        stream.synchronize()
        g.replay()
        stream.synchronize()
        assert_same_selection(gi.cpu().numpy(), gv.cpu().numpy(), oi, ov,
                              where=f"graph seed {seed} replay {rep}")
        topk.topk_ragged(s2, o2, l2, n2, K2, ei, ev, ws, stream)
        stream.synchronize()
        assert_same_selection(ei.cpu().numpy(), ev.cpu().numpy(), oi2, ov2,
                              where=f"eager mix between replays {rep}")
    del g


@pytest.mark.parametrize("K", [1, 3, 7168, 16384])
def test_mixed_call_extreme_k(topk, K):
    """Mixed rows at the ends of the K range (a few outputs per row; a K at and
    past the LDS frontier, 16384 at most 300 rows): selections and traces."""
    wl = mixed_workload(K % 97)
    n = wl.n_rows if K <= 8192 else min(wl.n_rows, 300)
    wl = W.Workload(wl.name, wl.scores, wl.row_offsets[:n].copy(), wl.row_lengths[:n].copy(),
                    K, "")
    gt, st = parity(topk, wl, where=f"mixed rows, K {K}", per_k=True)
    say("routes", st)
    assert st["errors"] == 0


@pytest.mark.parametrize("seed", range(3))
def test_mixed_call_random_policy(topk, seed):
    """Mixed calls under a random valid policy (stride 1 to 4096, any margins,
    including a nested target below the primary one, any sampling floor and
    frontier capacity): selections and traces."""
    rng = np.random.default_rng(7000 + seed)
    wl = mixed_workload(seed)
    pol = topk.default_policy()
    pol.s_log2 = int(rng.integers(0, 13))
    pol.rho_num, pol.rho_den = int(rng.integers(1, 9)), int(rng.integers(1, 5))
    pol.rho1_num, pol.rho1_den = int(rng.integers(1, 9)), int(rng.integers(1, 5))
    pol.l_samp_min = int(rng.choice([0, 1024, 8192, 65536, -1, -4, -16]))
    pol.cap = int(rng.choice([1, 100, 2048, 4095, 6144]))
    say("policy", pol.as_dict())
    gt, st = parity(topk, wl, policy=pol, where=f"mixed seed {seed}, random policy")
    say("routes", st)
    assert st["errors"] == 0


def shaped_workload(seed, n):
    """n rows of random kinds and lengths (about 15 M elements in all; up to
    700K per row when n <= 64), some lengths negative (read as 0), some rows
    overlapping earlier ones in the buffer."""
    rng = np.random.default_rng(12000 + seed)
    K = int(rng.choice([1, 16, 256, 2048, 4096]))
    mean = max(64, 30_000_000 // max(n, 1) // 2)
    lens = rng.integers(0, 2 * mean, n).astype(np.int64)
    if n <= 64:
        lens[:] = rng.integers(0, 700000, n)
    lens[rng.random(n) < 0.03] = -int(rng.integers(1, 100))
    pos, parts, offs = 0, [], np.zeros(n, np.int64)
    for r in range(n):
        L = max(int(lens[r]), 0)
        if r > 0 and pos > 0 and rng.random() < 0.1:
            offs[r] = int(rng.integers(0, pos))
            need = offs[r] + L - pos
            if need > 0:
                parts.append(rng.standard_normal(need).astype(np.float32))
                pos += need
            continue
        gap = int(rng.integers(0, 5))
        parts.append(np.zeros(gap, np.float32))
        pos += gap
        x = mixed_row(rng, KINDS[int(rng.integers(0, len(KINDS)))], L,
                      int(format(r % 128, "07b")[::-1], 2))
        parts.append(x)
        offs[r] = pos
        pos += x.size
    buf = np.concatenate(parts + [np.zeros(1, np.float32)]).astype(np.float32)
    return W.Workload(f"shape n={n}", buf, offs, lens.astype(np.int32), K, "")


@pytest.mark.parametrize("n", [1, 513, 16385])
def test_call_shapes(topk, n):
    """One row; one row past the split plan's limit (the item table); one row
    past the item table's (index order), with negative lengths and rows that
    overlap others in the buffer."""
    wl = shaped_workload(n, n)
    gt, st = parity(topk, wl, where=wl.name, per_k=True)
    say("routes", st)
    assert st["errors"] == 0


@pytest.mark.parametrize("seed", range(2))
def test_concurrent_calls_with_separate_workspaces(topk, seed):
    """Two mixed calls on two streams, each with its own workspace, launched
    back to back three times so that they overlap on the GPU: both equal the
    oracle every time."""
    import torch

    import oracle
    from tests.gpu_util import assert_same_selection, device_arrays

    streams = (torch.cuda.Stream(), torch.cuda.Stream())
    calls = []
    for w, st in zip((mixed_workload(seed), mixed_workload(seed + 5000)), streams):
        with torch.cuda.stream(st):
            s, o, l = device_arrays(w)
            ws = topk.alloc_workspace(w.n_rows, w.K, torch.device("cuda", 0), st)
            gi = torch.full((w.n_rows, w.K), -9, dtype=torch.int32, device="cuda")
            gv = torch.full((w.n_rows, w.K), 9.0, dtype=torch.float32, device="cuda")
        ref = oracle.topk_ragged(w.scores, w.row_offsets, w.row_lengths, w.K)
        calls.append((w, st, s, o, l, ws, gi, gv, ref))
    torch.cuda.synchronize()
    say("concurrent", [(c[0].n_rows, c[0].K) for c in calls])
    for rep in range(3):
        for w, st, s, o, l, ws, gi, gv, _ in calls:
            topk.topk_ragged(s, o, l, w.n_rows, w.K, gi, gv, ws, st)
        torch.cuda.synchronize()
        for w, st, s, o, l, ws, gi, gv, (oi, ov) in calls:
            assert_same_selection(gi.cpu().numpy(), gv.cpu().numpy(), oi, ov,
                                  where=f"{w.name}, concurrent, rep {rep}")


@pytest.mark.parametrize("shift", [1, 2, 3])
def test_mixed_call_misaligned_scores_pointer(topk, shift):
    """The scores pointer itself 4, 8 or 12 bytes past a 16-byte boundary (a
    slice of a larger buffer), on top of the rows' own odd offsets."""
    import torch

    import oracle
    from tests.gpu_util import assert_same_selection, run_hip

    wl = mixed_workload(20 + shift)
    big = torch.zeros(wl.scores.size + 4, dtype=torch.float32, device="cuda")
    big[shift:shift + wl.scores.size] = torch.from_numpy(wl.scores).cuda()
    s = big[shift:shift + wl.scores.size]
    assert s.data_ptr() % 16 == 4 * shift
    o = torch.from_numpy(wl.row_offsets).cuda()
    l = torch.from_numpy(wl.row_lengths).cuda()
    say("scores pointer +", 4 * shift, "bytes: rows", wl.n_rows, "K", wl.K)
    gi, gv, _, st = run_hip(s, o, l, wl.K, topk.policy_for_k(wl.K), trace=False)
    oi, ov = oracle.topk_ragged(wl.scores, wl.row_offsets, wl.row_lengths, wl.K)
    assert_same_selection(gi, gv, oi, ov, where=f"scores pointer +{4 * shift} B")
    assert st["errors"] == 0
