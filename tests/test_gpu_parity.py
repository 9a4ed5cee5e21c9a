"""GPU parity: the HIP path through the C-ABI against the CPU oracle.

Final selections are compared per row as (index, value-bits) sets with the
plain-definition oracle (bit-exact); per-row route traces are compared with
the oracle's step-by-step model (integer-exact).  Every case prints its name
before touching the GPU.
"""
import os

import numpy as np
import pytest

import oracle
from paper_2609_08450_amd import workloads as W
from tests.gpu_util import assert_same_selection, device_arrays, oracle_policy_of, run_hip
from tests.invariants import check_row

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def topk():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2609_08450_amd import topk as T

    T.lib()
    return T


def say(*a):
    print("[case]", *a, flush=True)


def parity(topk, wl, policy=None, trace=True, where="", per_k=False):
    """per_k: call without a policy (the library's topk_ragged_policy_for_k)."""
    import torch

    say(where or wl.name, "rows", wl.n_rows, "sum L", wl.total_len, "K", wl.K)
    s, o, l = device_arrays(wl)
    pol = topk.policy_for_k(wl.K) if per_k else (policy or topk.default_policy())
    gi, gv, gt, st = run_hip(s, o, l, wl.K, None if per_k else pol, trace)
    oi, ov = oracle.topk_ragged(wl.scores, wl.row_offsets, wl.row_lengths, wl.K)
    assert_same_selection(gi, gv, oi, ov, where=where or wl.name)
    if trace:
        _, _, mt = oracle.route_model(wl.scores, wl.row_offsets, wl.row_lengths, wl.K,
                                      oracle_policy_of(pol, wl.K))
        bad = np.nonzero(np.any(gt != mt, axis=1))[0]
        assert bad.size == 0, (f"{where}: trace differs on {bad.size} rows, first row {bad[0]}: "
                               f"gpu {gt[bad[0]].tolist()} oracle {mt[bad[0]].tolist()}")
    assert st["errors"] == 0
    del s, o, l
    torch.cuda.synchronize()
    return gt, st


# ------------------------------------------------------- building blocks --

def test_cutoffs_match_oracle(topk):
    import torch

    say("cutoffs")
    out = torch.zeros(2048, dtype=torch.int32, device="cuda")
    topk.debug_cutoffs(out)
    got = out.cpu().numpy().view(np.uint32)
    assert np.array_equal(got, oracle.cutoffs())


def test_coarse_map_matches_oracle(topk):
    import torch

    say("coarse map")
    top = np.arange(0, 1 << 19, dtype=np.uint32) << 13
    low = np.array([0, 1, 0x0FFF, 0x1000, 0x1001, 0x1FFF], np.uint32)
    pats = (top[:, None] | low[None, :]).ravel()
    rng = np.random.default_rng(5)
    pats = np.concatenate([pats, rng.integers(0, 1 << 32, 4_000_000, dtype=np.uint64).astype(np.uint32)])
    x = pats.view(np.float32)
    x = x[~np.isnan(x)]
    xd = torch.from_numpy(x).cuda()
    out = torch.empty(x.size, dtype=torch.int16, device="cuda")
    topk.debug_coarse(xd, out)
    got = out.cpu().numpy().view(np.uint16).astype(np.uint32)
    want = oracle.coarse(x)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(hex(int(x[i].view(np.uint32))), int(got[i]), int(want[i])) for i in bad[:5]]


# ---------------------------------------------------------- workloads ----

@pytest.mark.parametrize("cfg", [1, 2, 4, 5])
@pytest.mark.parametrize("per_k", [False, True], ids=["evaluated", "per-K"])
def test_parity_config(topk, cfg, per_k):
    """Every row of the config, selections and route traces.  per-K is the
    production call (no policy: topk_ragged_policy_for_k), which at K = 256
    routes config 1's rows differently from the evaluated constants."""
    wl = W.make(cfg)
    gt, st = parity(topk, wl, where=f"config {cfg} ({wl.name})", per_k=per_k)
    say("routes", st)


def test_parity_adversarial_recovery(topk):
    wl = W.adversarial_recovery()
    gt, st = parity(topk, wl)
    assert st["exact_underfill"] > 0 and st["band"] + st["exact_underfill"] > 0


def test_parity_chunked_prefill_all_rows(topk):
    """The full 4096 x 131072 causal block on the GPU, called as production
    calls it (no policy); every row's selection and route trace against the
    oracle (its OpenMP threads over the rows of the host copy)."""
    import torch

    say("chunked prefill 4096 rows (device-built scores)")
    s, offs, lens = W.chunked_prefill_device("cuda")
    n, K = lens.size, 2048
    o = torch.from_numpy(offs).cuda()
    l = torch.from_numpy(lens).cuda()
    gi, gv, gt, st = run_hip(s, o, l, K, None, True)
    host = s.reshape(-1).cpu().numpy()
    del s
    torch.cuda.synchronize()
    say("oracle over all rows")
    oi, ov = oracle.topk_ragged(host, offs, lens, K)
    assert_same_selection(gi, gv, oi, ov, where="chunked prefill")
    _, _, mt = oracle.route_model(host, offs, lens, K, oracle_policy_of(topk.policy_for_k(K), K))
    bad = np.nonzero(np.any(gt != mt, axis=1))[0]
    assert bad.size == 0, (f"chunked prefill: trace differs on {bad.size} rows, first row {bad[0]}: "
                           f"gpu {gt[bad[0]].tolist()} oracle {mt[bad[0]].tolist()}")
    assert st["errors"] == 0 and st["direct"] == 0
    say("routes", st)


# -------------------------------------------------------- forced routes --

def _mixed(K=2048):
    rng = np.random.default_rng(11)
    rows = []
    for L in (K - 1, K, K + 1, 5000, 9000, 30000, 70000, 140000, 300000):
        x = rng.standard_normal(L).astype(np.float32)
        rows.append(x)
        rows.append(np.round(x * 3).astype(np.float32))          # heavy ties
    rows.append(np.full(20000, 0.25, np.float32))                # all equal, > cap
    rows.append(np.where(rng.random(50000) < 0.5, -np.inf, 1.0).astype(np.float32))
    buf = np.concatenate(rows)
    lens = np.array([r.size for r in rows], np.int32)
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    return W.Workload("mixed", buf, offs, lens, K, "")


@pytest.mark.parametrize("name,kw", [
    ("default", {}),
    ("all exact", {"l_samp_min": 1 << 30}),
    ("small cap", {"cap": 3000}),
    ("tiny cap", {"cap": 600}),
    ("underfill", {"rho_num": 1, "rho_den": 2, "rho1_num": 3, "rho1_den": 4}),
    ("no band margin", {"rho_num": 1, "rho_den": 1, "rho1_num": 1, "rho1_den": 1}),
    ("nested target below", {"rho_num": 5, "rho_den": 2, "rho1_num": 5, "rho1_den": 4}),
    ("stride 64", {"s_log2": 6, "l_samp_min": 4096}),
    ("stride 1", {"s_log2": 0, "l_samp_min": 4096}),
    ("stride 4096", {"s_log2": 12, "l_samp_min": 0}),
])
def test_forced_routes(topk, name, kw):
    pol = topk.default_policy()
    for k, v in kw.items():
        setattr(pol, k, v)
    for wl in (_mixed(), W.adversarial(n_rows=96)):
        parity(topk, wl, policy=pol, where=f"{wl.name} / {name}")


# --------------------------------------------------------- random sweep --

def _random_workload(seed):
    """Rows of random lengths (a third at most K) and value families (normal,
    heavy ties, constant, -inf mix, decode mixture), seeded; n_rows alternates
    between call sizes that split rows and ones that do not."""
    rng = np.random.default_rng(2600 + seed)
    K = int([1, 5, 64, 300, 1024, 2048, 777, 2048][seed % 8])
    n_rows = int([7, 50, 700, 33, 500, 90, 400, 12][seed % 8])
    rows = []
    for r in range(n_rows):
        if rng.random() < 0.3:
            L = int(rng.integers(0, K + 1))
        else:
            L = int(np.exp(rng.uniform(np.log(K + 1), np.log(60000))))
        fam = int(rng.integers(0, 5))
        if fam == 0:
            x = rng.standard_normal(L).astype(np.float32)
        elif fam == 1:
            x = np.round(rng.standard_normal(L) * 4).astype(np.float32)
        elif fam == 2:
            x = np.full(L, np.float32(rng.standard_normal()), np.float32)
        elif fam == 3:
            x = rng.standard_normal(L).astype(np.float32)
            x[rng.random(L) < 0.4] = -np.inf
        else:
            x = W.decode_mixture_row(rng, L)
        rows.append(x.astype(np.float32))
    lens = np.array([r.size for r in rows], np.int32)
    offs = np.zeros(n_rows, np.int64)
    offs[1:] = np.cumsum(lens[:-1])
    buf = np.concatenate(rows) if rows else np.zeros(0, np.float32)
    return W.Workload(f"random{seed}", buf, offs, lens, K, "")


@pytest.mark.parametrize("seed", range(8))
def test_random_sweep(topk, seed):
    wl = _random_workload(seed)
    pol = topk.default_policy()
    choice = seed % 4
    if choice == 1:
        pol.cap = max(1, min(6144, 3 * wl.K // 2))
    elif choice == 2:
        pol.s_log2, pol.l_samp_min = 6, 0
    elif choice == 3:
        pol.rho_num, pol.rho_den, pol.rho1_num, pol.rho1_den = 1, 1, 5, 4
    parity(topk, wl, policy=pol, where=f"random{seed}/policy{choice}")


# ----------------------------------------------------------- edge cases --

def _edge_workload():
    rng = np.random.default_rng(13)
    sub1 = np.array([1], np.uint32).view(np.float32)[0]
    specials = np.array([0.0, -0.0, np.inf, -np.inf, sub1, -sub1, 1.0, -1.0], np.float32)
    rows = [np.zeros(0, np.float32), rng.standard_normal(1).astype(np.float32),
            rng.standard_normal(255).astype(np.float32), rng.standard_normal(256).astype(np.float32),
            rng.standard_normal(257).astype(np.float32),
            specials[rng.integers(0, 8, 5000)],
            specials[rng.integers(0, 8, 40000)],
            np.full(9000, -np.inf, np.float32),
            np.full(9000, -0.0, np.float32),
            np.concatenate([np.full(4000, 0.0, np.float32), np.full(6000, -0.0, np.float32)]),
            (rng.standard_normal(33333) * 1e-40).astype(np.float32)]  # subnormals
    lens = [r.size for r in rows] + [-5]
    rows.append(np.zeros(0, np.float32))
    # unaligned packing: odd gaps between rows
    parts, offs, pos = [], [], 0
    for r in rows:
        gap = int(rng.integers(0, 4))
        parts.append(rng.standard_normal(gap).astype(np.float32))
        pos += gap
        offs.append(pos)
        parts.append(r)
        pos += r.size
    buf = np.concatenate(parts)
    return W.Workload("edges", buf, np.array(offs, np.int64), np.array(lens, np.int32), 256, "")


def test_edge_rows(topk):
    wl = _edge_workload()
    parity(topk, wl)
    import torch

    s, o, l = device_arrays(wl)
    gi, gv, _, _ = run_hip(s, o, l, wl.K, topk.default_policy(), False)
    for r in range(wl.n_rows):
        check_row(wl.row(r), wl.K, gi[r], gv[r], f"edge row {r}")


def test_padded_pitch_rows(topk):
    rng = np.random.default_rng(17)
    n, pitch = 48, 70001
    buf = rng.standard_normal(n * pitch).astype(np.float32)
    lens = rng.integers(0, pitch + 1, n).astype(np.int32)
    wl = W.Workload("pitch", buf, (np.arange(n) * pitch).astype(np.int64), lens, 2048, "")
    parity(topk, wl)


def test_long_tie_row_uses_index_digits(topk):
    """2.5M equal values: the boundary bin exceeds the frontier (re-read path)
    and the tie is broken on all three index digits."""
    rng = np.random.default_rng(19)
    a = np.full(2_500_000, 0.75, np.float32)
    b = rng.standard_normal(3_000_000).astype(np.float32)
    b[rng.choice(b.size, 3000, replace=False)] = 9.0                    # 3000 ties at the top
    buf = np.concatenate([a, b])
    wl = W.Workload("long ties", buf, np.array([0, a.size], np.int64),
                    np.array([a.size, b.size], np.int32), 2048, "")
    gt, st = parity(topk, wl)
    assert st["reread"] >= 1


def _reread_rows(rng, L=131072):
    """Rows whose boundary coarse bin holds more entries than the frontier, so
    that the re-read path resolves it (K = 2048, 1500 to 1000 clear winners
    above the bin):
      keys+ties  distinct keys above a 10000-fold tie inside the bin, then
                 distinct keys below it: key rounds, then index rounds
      keys only  8000 distinct keys in one bin: key rounds end the search
      -inf       1000 finite values and 200 of -1e30 above 129K of -inf
      +inf bin   +inf, 1e10 and values past the FP16 range in bin 0
      zero bin   FP32 subnormals and tiny values above 20000 of +0.0, with
                 20000 of -0.0 (the next bin) and negatives below"""
    def base(mean=-3.0):
        return rng.normal(mean, 0.5, L).astype(np.float32)

    def put(x, vals):
        x[rng.choice(L, len(vals), replace=False)] = np.asarray(vals, np.float32)
        return x

    rows = {}
    x = base()
    # 1500 clear winners; bin of [2.0, 2.0625) (FP16 bin of 32 values at ulp 2^-9)
    pos = rng.choice(L, 1500 + 300 + 10000 + 2000, replace=False)
    x[pos[:1500]] = rng.uniform(5.0, 9.0, 1500).astype(np.float32)
    x[pos[1500:1800]] = rng.uniform(2.0400, 2.0600, 300).astype(np.float32)
    x[pos[1800:11800]] = np.float32(2.0390625)
    x[pos[11800:]] = rng.uniform(2.0005, 2.0380, 2000).astype(np.float32)
    rows["keys+ties"] = x
    x = base()
    pos = rng.choice(L, 1500 + 8000, replace=False)
    x[pos[:1500]] = rng.uniform(5.0, 9.0, 1500).astype(np.float32)
    x[pos[1500:]] = rng.uniform(2.0005, 2.0600, 8000).astype(np.float32)
    rows["keys only"] = x
    x = np.full(L, -np.inf, np.float32)
    rows["-inf"] = put(put(x, rng.standard_normal(1000)), np.full(200, -1e30))
    x = base()
    vals = np.concatenate([np.full(3000, np.inf), np.full(3000, 1e10),
                           rng.uniform(65600.0, 1e9, 4000)])
    rows["+inf bin"] = put(x, vals)
    x = base()
    pos = rng.choice(L, 1000 + 300 + 20000 + 20000, replace=False)
    x[pos[:1000]] = rng.uniform(1.0, 3.0, 1000).astype(np.float32)
    tiny = np.concatenate([np.frombuffer(rng.integers(1, 1 << 23, 150, dtype=np.uint32).tobytes(),
                                         np.float32), rng.uniform(1e-12, 1e-9, 150)])
    x[pos[1000:1300]] = tiny.astype(np.float32)
    x[pos[1300:21300]] = np.float32(0.0)
    x[pos[21300:]] = np.float32(-0.0)
    rows["zero bin"] = x
    return rows


@pytest.mark.parametrize("item_table", [False, True], ids=["split-plan", "item-table"])
def test_reread_windows(topk, item_table):
    """The re-read path's key and index windows, bit-exact with the oracle in
    both kernel instances (a call of a few rows, and one of more rows than
    resident workgroups, run from the item table)."""
    rng = np.random.default_rng(23)
    rows = list(_reread_rows(rng).values())
    if item_table:
        # 600 rows: the re-read rows among short rows of the direct and exact routes
        short = [rng.standard_normal(int(n)).astype(np.float32)
                 for n in rng.integers(100, 6000, 600 - len(rows))]
        rows = short[:300] + rows + short[300:]
    lens = np.array([r.size for r in rows], np.int32)
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    wl = W.Workload("re-read windows", np.concatenate(rows), offs, lens, 2048, "")
    gt, st = parity(topk, wl, where=f"re-read windows, item table {item_table}")
    say("routes", st)
    assert st["reread"] >= 5


@pytest.mark.parametrize("kind", ["clustered", "block"])
def test_decode_ties(topk, kind):
    """Decode-shaped batches with heavy ties (the rows of bench.py's ties
    ablation): every row's selection and trace, re-read rows included."""
    wl = W.decode_ties(kind)
    gt, st = parity(topk, wl, where=f"decode ties {kind}")
    say("routes", st)
    assert st["reread"] >= (64 if kind == "block" else 1)


def test_zero_rows_noop(topk):
    import torch

    say("zero rows")
    ws = topk.alloc_workspace(4, 16)
    e = torch.empty(0, device="cuda")
    topk.topk_ragged(e, torch.empty(0, dtype=torch.int64, device="cuda"),
                     torch.empty(0, dtype=torch.int32, device="cuda"), 0, 16,
                     torch.empty(0, dtype=torch.int32, device="cuda"), e, ws)
    torch.cuda.synchronize()


def test_workspace_too_small_is_flagged(topk):
    import torch

    wl = W.decode(n_rows=8)
    say("workspace for 4 rows, call with 8")
    s, o, l = device_arrays(wl)
    ws = topk.alloc_workspace(4, wl.K)
    gi, gv, _, st = run_hip(s, o, l, wl.K, None, False, ws=ws)
    assert st["errors"] == 1
    assert np.all(gi == -1) and np.all(np.isneginf(gv))


def test_repeated_calls_are_stable(topk):
    """Split rows reuse per-row state: 30 calls on one workspace must agree."""
    import torch

    wl = W.decode()
    say("decode x30")
    s, o, l = device_arrays(wl)
    ws = topk.alloc_workspace(wl.n_rows, wl.K)
    oi, ov = oracle.topk_ragged(wl.scores, wl.row_offsets, wl.row_lengths, wl.K)
    for it in range(30):
        gi, gv, _, st = run_hip(s, o, l, wl.K, None, False, ws=ws)
        assert_same_selection(gi, gv, oi, ov, where=f"decode call {it}")


def test_graph_capture_and_replay(topk):
    """Four calls (three workloads, one of them with the order pre-pass)
    captured in one HIP graph, replayed with host work and synchronisation
    between replays; every replay must match the eager results."""
    import torch

    wa, wb, wc = W.decode(), W.adversarial(n_rows=128), W.adversarial(n_rows=1024)
    say("graph replay")
    sa, oa, la = device_arrays(wa)
    sb, ob, lb = device_arrays(wb)
    sc, oc, lc = device_arrays(wc)
    K = 2048
    wsa = topk.alloc_workspace(wa.n_rows, K)
    wsb = topk.alloc_workspace(wb.n_rows, K)
    wsc = topk.alloc_workspace(wc.n_rows, K)

    def outs_for(w):
        return (torch.empty((w.n_rows, K), dtype=torch.int32, device="cuda"),
                torch.empty((w.n_rows, K), dtype=torch.float32, device="cuda"))

    outs = [outs_for(wa), outs_for(wb), outs_for(wa), outs_for(wc)]
    # the 1024-row call has more rows than 2 x CUs: the order pre-pass and the
    # main kernel are both captured
    calls = [(sa, oa, la, wa.n_rows, wsa), (sb, ob, lb, wb.n_rows, wsb),
             (sa, oa, la, wa.n_rows, wsa), (sc, oc, lc, wc.n_rows, wsc)]
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for (s, o, l, n, ws), (oi, ov) in zip(calls, outs):       # warm-up, eager
            topk.topk_ragged(s, o, l, n, K, oi, ov, ws, stream)
    stream.synchronize()
    eager = [(oi.cpu().numpy(), ov.cpu().numpy()) for oi, ov in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for (s, o, l, n, ws), (oi, ov) in zip(calls, outs):
            topk.topk_ragged(s, o, l, n, K, oi, ov, ws, torch.cuda.current_stream())
    for rep in range(10):
        for oi, ov in outs:
            oi.fill_(-9)
            ov.fill_(0.5)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for j, (oi, ov) in enumerate(outs):
            assert_same_selection(oi.cpu().numpy(), ov.cpu().numpy(), *eager[j],
                                  where=f"replay {rep} call {j}")
    ri, rv = oracle.topk_ragged(wa.scores, wa.row_offsets, wa.row_lengths, K)
    assert_same_selection(*eager[0], ri, rv, where="eager vs oracle")
    ri, rv = oracle.topk_ragged(wc.scores, wc.row_offsets, wc.row_lengths, K)
    assert_same_selection(*eager[3], ri, rv, where="eager vs oracle (1024 rows)")


def test_outputs_not_16_byte_aligned(topk):
    """Output rows that start off the 16-byte grid (4-byte aligned views)
    take the 4-byte store path of the staged write-out."""
    import torch

    wl = W.decode(n_rows=12)
    say("decode 12 rows, outputs offset by one element")
    s, o, l = device_arrays(wl)
    n, K = wl.n_rows, wl.K
    ws = topk.alloc_workspace(n, K)
    bi = torch.full((n * K + 1,), -7, dtype=torch.int32, device="cuda")
    bv = torch.full((n * K + 1,), 7.0, dtype=torch.float32, device="cuda")
    oi_d, ov_d = bi[1:], bv[1:]
    assert oi_d.data_ptr() % 16 != 0
    topk.topk_ragged(s, o, l, n, K, oi_d, ov_d, ws)
    torch.cuda.synchronize()
    assert int(bi[0]) == -7 and float(bv[0]) == 7.0   # nothing written before the rows
    gi = oi_d.view(n, K).cpu().numpy()
    gv = ov_d.view(n, K).cpu().numpy()
    oi, ov = oracle.topk_ragged(wl.scores, wl.row_offsets, wl.row_lengths, K)
    assert_same_selection(gi, gv, oi, ov, where="unaligned outputs")


def test_shared_view_rows(topk):
    """Split rows whose view is large enough to be shared by their segments
    (each histograms the view positions in its own range, the last merges):
    the boundaries, routes and selections must equal the oracle's."""
    rng = np.random.default_rng(23)
    lens = np.array([524288, 700001, 1048576, 600000, 530000], np.int32)
    rows = []
    for i, L in enumerate(lens):
        x = W.decode_mixture_row(rng, int(L))
        if i == 3:
            x = np.round(x * 8.0).astype(np.float32) / 8.0      # heavy ties
        rows.append(x.astype(np.float32))
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    for K in (2048, 300):
        wl = W.Workload(f"shared view K={K}", np.concatenate(rows), offs, lens, K, "")
        parity(topk, wl)


@pytest.mark.parametrize("K", [1, 7, 100, 256, 383, 384, 512, 1000, 1024, 1600, 2047, 2500,
                               2560, 3000, 4096, 4351, 4352, 6000, 8192, 16384])
def test_parity_per_k_policy(topk, K):
    """Calls without a policy use the per-K constants (topk_ragged_policy_for_k):
    decode-mixture rows around the sampling floor and up to 131072 elements,
    selections and per-row routes against the oracle under that policy.  From
    K = 8192 (past the on-chip frontier) a row of 200000 equal values is
    added: its boundary bin holds more entries than the frontier, so the
    re-read path runs at large K too."""
    rng = np.random.default_rng(1000 + K)
    lens = sorted({max(1, K - 1), K + 1, 4 * K - 1, 4 * K, 4 * K + 7, 10 * K + 3, 16384, 40000,
                   90001, 131072})
    rows = [W.decode_mixture_row(rng, int(L)).astype(np.float32) for L in lens]
    if K >= 8192:
        rows.append(np.full(200000, 0.5, np.float32))
        lens.append(200000)
    lens = np.array(lens, np.int32)
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    wl = W.Workload(f"per-K policy K={K}", np.concatenate(rows), offs, lens, K, "")
    gt, st = parity(topk, wl, per_k=True)
    say("routes", st)
    if K >= 4352:
        assert st["primary"] + st["band"] == 0
    if K >= 8192:
        assert st["reread"] >= 1


@pytest.mark.parametrize("n", [400, 600])
def test_single_workgroup_rows_with_an_overflowed_region(topk, n):
    """Rows whose admitted tail lies in positions one wave streams: that
    wave's region overflows, so C(tau0) comes from a coarse histogram (a
    re-read of the row; in a call run from the item table, 600 rows of one
    workgroup each, Phase 2 goes on and counts the hits its region cannot
    keep); rows whose proposal certifies re-collect their frontier,
    overflowing ones reuse the histogram for the exact route."""
    rng = np.random.default_rng(31)
    L = 24576
    hot = (np.arange(L) % 2048) < 256   # the positions of wave 0 in every chunk
    rows = []
    for i in range(n):
        x = W.decode_mixture_row(rng, L).astype(np.float32)
        if i % 4 == 0:                   # C(tau0) within the frontier: primary
            x[hot] = rng.normal(4.0, 0.1, int(hot.sum())).astype(np.float32)
        elif i % 4 == 1:                 # the view sees only low values: overflow
            x[hot] = rng.normal(4.0, 0.1, int(hot.sum())).astype(np.float32)
            phase = int(format(i % 128, "07b")[::-1], 2)   # the row's view phase
            x[phase::128] = rng.normal(-2.0, 1.0, x[phase::128].size).astype(np.float32)
        rows.append(x)
    lens = np.full(n, L, np.int32)
    offs = (np.arange(n, dtype=np.int64) * L)
    wl = W.Workload("one-wave tails", np.concatenate(rows), offs, lens, 2048, "")
    gt, st = parity(topk, wl)
    say("routes", st)
    assert st["primary"] > 0 and st["exact_overflow"] > 0


def test_split_rows_with_an_overflowed_region(topk):
    """Rows split across workgroups (a call of 48 rows) where some segments
    see their admitted tail in one wave's positions: those segments re-count
    by re-reading (both counts), the others publish per wave, and the
    finisher of a row with an incomplete segment re-collects or takes the
    exact route."""
    rng = np.random.default_rng(37)
    n = 48
    lens = rng.integers(40000, 131072, n).astype(np.int32)
    rows = []
    for i, L in enumerate(lens):
        x = W.decode_mixture_row(rng, int(L)).astype(np.float32)
        hot = np.nonzero((np.arange(L) % 2048) < 256)[0]
        if i % 3 == 0:      # a tail of ~2.5 K in wave-0 positions of one stretch
            sel = hot[(hot > L // 3) & (hot < L // 3 + 20000)]
            x[sel] = rng.normal(4.0, 0.1, sel.size).astype(np.float32)
        elif i % 3 == 1:    # too many candidates everywhere: overflow
            phase = int(format(i % 128, "07b")[::-1], 2)
            x[phase::128] = rng.normal(-2.0, 1.0, x[phase::128].size).astype(np.float32)
        rows.append(x)
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    wl = W.Workload("split one-wave tails", np.concatenate(rows), offs, lens, 2048, "")
    gt, st = parity(topk, wl)
    say("routes", st)
    assert st["exact_overflow"] > 0 and st["primary"] + st["band"] > 0


def test_many_rows_halves_the_long_ones(topk):
    """A call of more rows than the item target but within the resident
    workgroups (450 rows): rows longer than the mean are cut in two."""
    rng = np.random.default_rng(41)
    n = 450
    lens = np.where(rng.random(n) < 0.2, rng.integers(60000, 131072, n),
                    rng.integers(3000, 30000, n)).astype(np.int32)
    rows = [W.decode_mixture_row(rng, int(L)).astype(np.float32) for L in lens]
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    wl = W.Workload("many rows", np.concatenate(rows), offs, lens, 2048, "")
    gt, st = parity(topk, wl)
    say("routes", st)
    assert st["errors"] == 0


def _longest_first_workload(n):
    rng = np.random.default_rng(47 + n)
    if n <= 2000:
        lens = np.where(rng.random(n) < 0.15, rng.integers(100000, 200000, n),
                        rng.integers(0, 12000, n)).astype(np.int32)
        lens[rng.choice(n, 20, replace=False)] = 0
    else:
        lens = rng.integers(1, 4000, n).astype(np.int32)
    rows = [W.decode_mixture_row(rng, int(L)).astype(np.float32) for L in lens]
    place = rng.permutation(n)             # row place[j] is the j-th in the buffer
    offs = np.zeros(n, np.int64)
    offs[place] = np.concatenate([[0], np.cumsum(lens[place][:-1])])
    buf = np.concatenate([rows[r] for r in place])
    return W.Workload("longest first", buf, offs, lens, 2048, "")


@pytest.mark.parametrize("n", [1500, 16385])
def test_many_rows_run_longest_first(topk, n):
    """Calls whose rows each take one workgroup run them longest first
    (1500 rows, lengths from empty to 200K in random order, stored in the
    buffer in another order than their indices; the longest are cut into
    segments); above the order's row limit (16385 short rows) they run in
    index order.  Same selections either way."""
    gt, st = parity(topk, _longest_first_workload(n))
    say("routes", st)
    assert st["errors"] == 0


def _length_class(L):
    if L < 8:
        return max(int(L), 0)
    e = int(L).bit_length() - 1
    return e * 8 + ((int(L) >> (e - 3)) & 7)


@pytest.mark.parametrize("case", ["edge mix", "1500 rows"])
def test_item_table_cuts_the_longest_rows(topk, case):
    """The item table of a call with more rows than resident workgroups, read
    back from the workspace: rows longest first by length class; each row's
    segments consecutive items with the row's length and offset; the segment
    counts of the rule, P = min(64, L / 8192, ceil(L / S)) with S = max(8192,
    ceil(sum L / resident workgroups)) for the 1024 longest rows, kept down the
    order while the extra items fit the budget and the split rows the per-row
    state; split rows in slots 0, 1, 2, ...; the rest of the table empty."""
    import torch

    wl = W.make(5) if case == "edge mix" else _longest_first_workload(1500)
    n, K = wl.n_rows, wl.K
    say("item table", case, "rows", n)
    s, o, l = device_arrays(wl)
    ws = topk.alloc_workspace(n, K)
    run_hip(s, o, l, K, trace=False, ws=ws)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    extra, slots = min(2 * cus, 1024), 2 * cus
    split_rows = int(ws[:1024].cpu().numpy().view(np.uint32)[1])
    tab = ws[1024:1024 + 16 * (n + extra)].cpu().numpy().view(np.uint32).reshape(-1, 4)
    tab = tab.astype(np.int64)
    x, y, z, w = tab[:, 0], tab[:, 1], tab[:, 2], tab[:, 3]
    live = (x >> 31) == 0
    T = int(live.sum())
    assert live[:T].all() and not live[T:].any(), "empty items must follow the last segment"
    r, p, P = x & 0x3FFF, (x >> 14) & 63, ((x >> 20) & 63) + 1
    off, slot = z | ((w & 0xFF) << 32), w >> 8
    lens = wl.row_lengths.astype(np.int64)
    S = max(8192, -(-int(np.maximum(lens, 0).sum()) // slots))
    seen = np.zeros(n, bool)
    i, k, E, Ns, prev_cls = 0, 0, 0, 0, 1 << 30
    while i < T:
        row = int(r[i])
        assert not seen[row], f"row {row} listed twice"
        seen[row] = True
        Pi, Lr = int(P[i]), int(lens[row])
        for q in range(Pi):
            j = i + q
            assert (r[j], p[j], P[j], y[j], off[j], slot[j]) == \
                (row, q, Pi, Lr, wl.row_offsets[row], slot[i]), f"item {j}"
        c = _length_class(Lr)
        assert c <= prev_cls, f"rank {k}: class {c} after {prev_cls}"
        prev_cls = c
        want = 1
        if k < 1024 and 16384 <= Lr:
            want = min(64, Lr // 8192, -(-Lr // S))
        E, Ns = E + want - 1, Ns + (want > 1)
        kept = E <= extra and Ns <= split_rows
        assert Pi == (want if kept else 1), f"rank {k} row {row} L {Lr}: P {Pi}, rule {want}"
        if Pi > 1:
            assert slot[i] == Ns - 1
        i += Pi
        k += 1
    assert seen.all()
    assert T - n == int((P[:T][p[:T] == 0] - 1).sum()) <= extra
    say("split rows", int(((P[:T] > 1) & (p[:T] == 0)).sum()), "extra items", T - n, "S", S)
    assert (P[:T] > 1).any(), "the workload should cut some rows"


def test_segments_that_stop_waiting_build_the_view(topk):
    """With one poll allowed, split segments that do not see segment 0's
    boundaries at once build the whole view themselves (a small view, and a
    shared large one): same boundaries, routes and selections."""
    rng = np.random.default_rng(43)
    lens = np.array([524288, 600000, 90000, 131072, 40000, 70000], np.int32)
    rows = [W.decode_mixture_row(rng, int(L)).astype(np.float32) for L in lens]
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    wl = W.Workload("spin limit 1", np.concatenate(rows), offs, lens, 2048, "")
    topk.debug_set_spin_limit(1)
    try:
        gt, st = parity(topk, wl)
    finally:
        topk.debug_set_spin_limit(0)
    say("routes", st)
    assert st["wait_fallback"] > 0


def test_item_table_caps_a_row_at_64_segments(topk):
    """A call of 600 rows, one of 8M elements (an eighth of the call's
    length and more), two of 2M and short ones: the longest row gets the cap
    of 64 segments (its own ceil(L / S) is larger), the 2M rows what the
    rule gives, and every selection and trace still matches the oracle.  (The
    extra-item budget of 2 x CUs cannot bind: the cut rows' extra items sum to
    at most sum(L) / S <= 2 x CUs.)"""
    import torch

    rng = np.random.default_rng(59)
    n = 600
    lens = rng.integers(1000, 9000, n).astype(np.int32)
    big = rng.choice(n, 3, replace=False)
    lens[big[0]] = 8_000_000
    lens[big[1:]] = 2_000_000
    rows = [W.decode_mixture_row(rng, int(L)).astype(np.float32) for L in lens]
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    wl = W.Workload("segment cap", np.concatenate(rows), offs, lens, 2048, "")
    gt, st = parity(topk, wl)
    say("routes", st)
    s, o, l = device_arrays(wl)
    ws = topk.alloc_workspace(n, wl.K)
    run_hip(s, o, l, wl.K, trace=False, ws=ws)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    extra = min(2 * cus, 1024)
    tab = ws[1024:1024 + 16 * (n + extra)].cpu().numpy().view(np.uint32).reshape(-1, 4)
    tab = tab.astype(np.int64)
    first = ((tab[:, 0] >> 31) == 0) & (((tab[:, 0] >> 14) & 63) == 0)
    seg = dict(zip((tab[first, 0] & 0x3FFF).tolist(), (((tab[first, 0] >> 20) & 63) + 1).tolist()))
    S = max(8192, -(-int(lens.astype(np.int64).sum()) // (2 * cus)))
    say("segments", seg[int(big[0])], seg[int(big[1])], seg[int(big[2])], "S", S)
    assert seg[int(big[0])] == 64
    for r in big[1:]:
        assert seg[int(r)] == min(64, 2_000_000 // 8192, -(-2_000_000 // S))


def _split_exact_workload():
    """600 rows: 60 long ones (150K-250K, cut into segments by the item table)
    among short ones.  Long row kinds by i % 4: 0 a decode row (primary); 1
    the view residue N(-2, 1) (every segment overflows: the split exact
    route); 2 a tail of ~2.5 K in the positions of one wave in one stretch
    (a segment overflows, the row certifies: the route is abandoned); 3 low
    values, the view residue lower still, and 10000 copies of 1.0 (overflow
    with tau_star's bin beyond the frontier: abandoned for the re-read)."""
    rng = np.random.default_rng(53)
    n = 600
    lens = rng.integers(2000, 8000, n).astype(np.int32)
    longs = rng.choice(n, 60, replace=False)
    lens[longs] = rng.integers(150000, 250000, 60)
    rows = []
    kind = {int(r): j % 4 for j, r in enumerate(longs)}
    for i, L in enumerate(lens):
        L = int(L)
        x = W.decode_mixture_row(rng, L).astype(np.float32)
        phase = int(format(i % 128, "07b")[::-1], 2)
        k = kind.get(i, -1)
        if k == 1:
            x[phase::128] = rng.normal(-2.0, 1.0, x[phase::128].size).astype(np.float32)
        elif k == 2:
            hot = np.nonzero((np.arange(L) % 2048) < 256)[0]
            sel = hot[(hot > L // 3) & (hot < L // 3 + 20000)]
            x[sel] = rng.normal(4.0, 0.1, sel.size).astype(np.float32)
        elif k == 3:
            x = rng.normal(-3.0, 0.5, L).astype(np.float32)
            x[rng.choice(L, 10000, replace=False)] = 1.0
            x[phase::128] = rng.normal(-5.0, 1.0, x[phase::128].size).astype(np.float32)
        rows.append(x)
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    return W.Workload("split exact route", np.concatenate(rows), offs, lens, 2048, "")


@pytest.mark.parametrize("spin", [0, 1], ids=["waits", "one-poll"])
def test_split_exact_route(topk, spin):
    """Overflowing rows cut into segments take the exact route across their
    segments (histograms merged, tau_star published, each segment classifies
    its own range, the last refines); rows where it does not apply abandon it
    for the finisher.  With one poll allowed, segments stop waiting for
    tau_star and the last arrival classifies their ranges.  Same selections
    and traces as the oracle either way."""
    wl = _split_exact_workload()
    topk.debug_set_spin_limit(spin)
    try:
        gt, st = parity(topk, wl, where=f"split exact route, spin {spin}")
    finally:
        topk.debug_set_spin_limit(0)
    say("routes", st)
    assert st["exact_overflow"] > 0 and st["primary"] > 0 and st["reread"] > 0
    if spin:
        assert st["wait_fallback"] > 0


@pytest.mark.parametrize("cfg", [2, 5])
def test_read_ceiling_reads_every_score(topk, cfg):
    """The read-only ceiling kernel (the measurement's bound) visits every
    valid score of every row once: its per-row maximum key equals numpy's."""
    import torch

    wl = W.make(cfg)
    say("read ceiling", wl.name)
    s, o, l = device_arrays(wl)
    out = torch.zeros(wl.n_rows, dtype=torch.int32, device="cuda")
    ws = topk.alloc_workspace(wl.n_rows, wl.K)
    topk.debug_read_ceiling(s, o, l, wl.n_rows, wl.K, out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint32)
    want = np.zeros(wl.n_rows, np.uint32)
    for r in range(wl.n_rows):
        x = wl.row(r)
        if x.size:
            want[r] = oracle.asc32(x.view(np.uint32)).max()
    assert np.array_equal(got, want)


def test_rows_at_the_length_limit(topk):
    """Rows of exactly TOPK_L_MAX elements (2^30 - 33), at an aligned offset and
    at the worst misalignment (31 elements: the last of a 128-byte line, so
    the streamed range starts 31 elements before the row), whose Top-K is
    known by construction: K distinct positive values planted among negative
    ones.
    Both return exactly the planted (index, value) set.  A row one element
    longer is rejected on the device: -1 / -inf and one error count."""
    import re

    import torch

    text = open(os.path.join(ROOT, "include", "topk_ragged.h")).read()
    lmax = int(re.search(r"#define TOPK_L_MAX (0x[0-9A-Fa-f]+)", text).group(1), 16)
    K = 2048
    say("rows of", lmax, "elements")
    x = torch.rand(lmax + 32, device="cuda")
    x.add_(1.0).neg_()                            # every value in (-2, -1]
    rng = np.random.default_rng(71)
    pos = np.sort(rng.choice(np.arange(31, lmax, dtype=np.int64), K, replace=False))
    vals = (1.0 + rng.permutation(K) / 4096.0).astype(np.float32)
    x[torch.from_numpy(pos).cuda()] = torch.from_numpy(vals).cuda()
    offs = torch.tensor([0, 31, 0], dtype=torch.int64, device="cuda")
    lens = torch.tensor([lmax, lmax, lmax + 1], dtype=torch.int32, device="cuda")
    gi, gv, _, st = run_hip(x, offs, lens, K, trace=False)
    del x
    torch.cuda.empty_cache()
    want = {int(p): int(v) for p, v in zip(pos, vals.view(np.uint32))}
    for r, shift in ((0, 0), (1, 31)):
        got = {int(i) + shift: int(v) for i, v in zip(gi[r], gv[r].view(np.uint32))}
        assert got == want, f"row {r}: {len(set(got) ^ set(want))} positions differ"
    assert np.all(gi[2] == -1) and np.all(np.isneginf(gv[2]))
    assert st["errors"] == 1, st
    say("routes", st)
