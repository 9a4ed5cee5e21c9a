"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: expected values come from hand
derivations (tests/golden/worked_examples.json), numpy's IEEE float16
conversion, numpy sorting, pure-Python brute force, and closed forms.
"""
import itertools
import json
import math
import os
import struct

import numpy as np
import pytest

import oracle
from oracle import Policy
from paper_2609_08450_amd import workloads as W
from tests.invariants import check_row, reference_rank

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def f32(v):
    """Golden-file value -> np.float32 (hex strings are FP32 bit patterns)."""
    if isinstance(v, str):
        return np.array([int(v, 16)], np.uint32).view(np.float32)[0]
    return np.float32(v)


def asc_of_value(x):
    """Ascending key of one FP32 value, from numeric order (for golden cutoffs)."""
    return int(oracle.asc32(np.array([np.float32(x)]).view(np.uint32))[0])


@pytest.fixture(scope="module")
def golden():
    with open(GOLDEN) as fh:
        return json.load(fh)


# ------------------------------------------------------------ golden pins --

def test_golden_coarse(golden):
    for e in golden["coarse"]:
        x = f32(e["bits"]) if "bits" in e else np.float32(e["x"])
        assert int(oracle.coarse(np.array([x]))[0]) == e["c"], e


def test_golden_cutoffs(golden):
    cut = oracle.cutoffs()
    for e in golden["cutoffs"]:
        t = e["tau"]
        if "cut" in e:
            want = int(e["cut"], 16)
        elif "cut_value" in e:
            want = asc_of_value(e["cut_value"])
        else:
            want = asc_of_value(f32(e["cut_bits"]))
        assert int(cut[t]) == want, (t, hex(int(cut[t])), hex(want), e["why"])


def test_golden_plain(golden):
    for e in golden["plain"]:
        x = np.array([f32(v) for v in e["row"]], np.float32)
        K = e["K"]
        oi, ov = oracle.topk_ragged(x, [0], [x.size], K)
        if e.get("direct"):
            exp = list(range(x.size)) + [-1] * (K - x.size)
            assert oi[0].tolist() == exp
        else:
            assert sorted(oi[0].tolist()) == e["idx"], e
        assert np.array_equal(ov[0][oi[0] >= 0].view(np.uint32), x[oi[0][oi[0] >= 0]].view(np.uint32))


def test_golden_route(golden):
    for e in golden["route"]:
        x = np.array([f32(v) for v in e["row"]], np.float32)
        pol = oracle.default_policy(**e["policy"])
        oi, ov, tr = oracle.route_model(x, [0], [x.size], e["K"], pol)
        assert sorted(oi[0].tolist()) == e["idx"], (e["why"], oi[0])
        assert tr[0].tolist() == e["trace"], (e["why"], tr[0].tolist())


# ------------------------------------------------------ key transform ----

def _structured_patterns():
    """Bit patterns covering every exponent, both signs, the subnormal range,
    +/-0, +/-inf and the extremes of each binade; NaNs excluded."""
    rng = np.random.default_rng(1)
    hi = np.arange(0, 1 << 9, dtype=np.uint32) << 23          # sign + exponent
    lo = np.array([0, 1, 2, 0x3FFFFF, 0x400000, 0x7FFFFE, 0x7FFFFF], np.uint32)
    a = (hi[:, None] | lo[None, :]).ravel()
    b = rng.integers(0, 1 << 32, 200_000, dtype=np.uint64).astype(np.uint32)
    pats = np.unique(np.concatenate([a, b]))
    x = pats.view(np.float32)
    return pats[~np.isnan(x)]


def test_asc32_orders_like_numbers():
    pats = _structured_patterns()
    x = pats.view(np.float32)
    order = np.lexsort((~np.signbit(x), x.astype(np.float64)))  # numeric, -0 before +0
    keys = oracle.asc32(pats[order])
    assert np.all(np.diff(keys.astype(np.int64)) > 0)
    z = np.array([0x80000000, 0x00000000], np.uint32)
    assert oracle.asc32(z).tolist() == [0x7FFFFFFF, 0x80000000]


# ------------------------------------------------- FP16 projection -------

def test_fp16_rn_matches_numpy():
    # every sign/exponent/top-10-mantissa prefix with the rounding-relevant
    # low 13 bits at and around the half-way point, plus random patterns
    top = np.arange(0, 1 << 19, dtype=np.uint32) << 13
    low = np.array([0, 1, 0x0FFF, 0x1000, 0x1001, 0x1FFF], np.uint32)
    pats = (top[:, None] | low[None, :]).ravel()
    rng = np.random.default_rng(2)
    pats = np.concatenate([pats, rng.integers(0, 1 << 32, 1_000_000, dtype=np.uint64).astype(np.uint32)])
    x = pats.view(np.float32)
    x = x[~np.isnan(x)]
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).view(np.uint16)
    got = oracle.fp16_rn(x)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(hex(int(x[i].view(np.uint32))), hex(int(got[i])), hex(int(want[i]))) for i in bad[:5]]


def test_coarse_is_monotone_and_covers_bins():
    pats = _structured_patterns()
    x = pats.view(np.float32)
    order = np.lexsort((~np.signbit(x), x.astype(np.float64)))
    c = oracle.coarse(x[order]).astype(np.int64)
    # eq:method:coarse-order: a larger value never lands in a worse bin
    assert np.all(np.diff(c) <= 0)
    # the FP16 image of the non-NaN line spans bins c(+inf)=31 .. c(-inf)=2016
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16)
    h = h[~np.isnan(h)].astype(np.float32)
    ch = oracle.coarse(h)
    assert ch.min() == 31 and ch.max() == 2016
    counts = np.bincount(ch, minlength=2048)
    assert np.all(counts[32:2016] == 32)  # every interior bin groups 32 FP16 keys


def test_cutoffs_against_numpy_rounding():
    """cut[tau] is the first FP32 value (in ascending order) whose numpy FP16
    rounding lands in a bin <= tau: checked at cut and at its predecessor."""
    cut = oracle.cutoffs()
    def inv(u):  # ascending key -> value
        u = np.uint32(u)
        b = (u & np.uint32(0x7FFFFFFF)) if (u & np.uint32(0x80000000)) else ~u
        return np.array([b], np.uint32).view(np.float32)[0]
    def bin_numpy(v):
        with np.errstate(over="ignore"):
            h = int(np.array([v], np.float32).astype(np.float16).view(np.uint16)[0])
        return ((0x7FFF - h) >> 5) if h < 0x8000 else (h >> 5)
    for t in range(2048):
        u = int(cut[t])
        if u == 0xFFFFFFFF:
            assert t < 31
            continue
        assert bin_numpy(inv(u)) <= t
        if u > 0x007FFFFF:
            assert bin_numpy(inv(u - 1)) > t


# ----------------------------------------------- plain definition --------

SPECIAL = [0.0, -0.0, 1.0, -1.0, math.inf, -math.inf,
           struct.unpack("<f", struct.pack("<I", 1))[0],
           struct.unpack("<f", struct.pack("<I", 0x80000001))[0]]


def brute_force(row, K):
    """Pure-Python exact Top-K on numeric order (-0.0 below +0.0), lowest index first."""
    L = len(row)
    if L <= K:
        return list(range(L)) + [-1] * (K - L)
    key = lambda i: (-row[i], -math.copysign(1.0, row[i]), i)
    return sorted(sorted(range(L), key=key)[:K])


def test_plain_exhaustive_small_alphabet():
    alpha = [np.float32(v) for v in SPECIAL[:7]]
    for L in range(0, 5):
        for combo in itertools.product(alpha, repeat=L):
            row = np.array(combo, np.float32)
            for K in range(1, L + 3):
                oi, _ = oracle.topk_ragged(row, [0], [L], K)
                got = oi[0].tolist() if L <= K else sorted(oi[0].tolist())
                assert got == brute_force([float(v) for v in row], K), (row, K)


def test_plain_random_tiny_rows_vs_brute_force():
    rng = np.random.default_rng(3)
    for _ in range(300):
        L = int(rng.integers(1, 40))
        pool = np.array(SPECIAL + list(rng.standard_normal(6)), np.float32)
        row = pool[rng.integers(0, pool.size, L)]
        K = int(rng.integers(1, L + 3))
        oi, ov = oracle.topk_ragged(row, [0], [L], K)
        got = oi[0].tolist() if L <= K else sorted(oi[0].tolist())
        assert got == brute_force([float(v) for v in row], K)
        check_row(row, K, oi[0], ov[0])


def test_plain_ragged_layout_and_lexsort():
    rng = np.random.default_rng(4)
    lens = rng.integers(-3, 6000, 40).astype(np.int32)
    gaps = rng.integers(0, 7, 40)
    offs, pos = [], 0
    for L, g in zip(lens, gaps):
        pos += int(g)
        offs.append(pos)
        pos += max(0, int(L))
    buf = rng.standard_normal(pos + 5).astype(np.float32)
    buf[rng.random(buf.size) < 0.05] = -np.inf
    buf[rng.random(buf.size) < 0.05] = 0.5
    K = 700
    oi, ov = oracle.topk_ragged(buf, np.array(offs), lens, K)
    for r, (o, L) in enumerate(zip(offs, lens)):
        row = buf[o:o + max(0, int(L))]
        check_row(row, K, oi[r], ov[r], f"row {r}")
        if row.size > K:  # canonical order: exactly the lexsort order
            assert np.array_equal(oi[r], reference_rank(row)[:K])


# ---------------------------------------------------- route model -------

def test_phase_is_bit_reversal_permutation():
    assert [oracle.phase(r, 128) for r in (0, 1, 2, 3, 127, 128, 129)] == [0, 64, 32, 96, 127, 0, 64]
    for s in (1, 2, 4, 64, 128, 256):
        assert sorted(oracle.phase(r, s) for r in range(s)) == list(range(s))


def test_sample_ranks():
    assert oracle.sample_rank(2048, 3, 2, 128) == 24
    assert oracle.sample_rank(2048, 7, 4, 128) == 28
    assert oracle.sample_rank(256, 3, 2, 128) == 3
    assert oracle.sample_rank(256, 7, 4, 128) == 4


def _route_checks(wl, K, pol, rows=None):
    rows = range(wl.n_rows) if rows is None else rows
    sub = wl.subset(rows)
    oi, ov, tr = oracle.route_model(sub.scores, sub.row_offsets, sub.row_lengths, K, pol)
    pi, pv = oracle.topk_ragged(sub.scores, sub.row_offsets, sub.row_lengths, K)
    s = pol.s
    q0 = math.ceil(pol.rho_num * K / (pol.rho_den * s))
    q1 = max(q0, math.ceil(pol.rho1_num * K / (pol.rho1_den * s)))  # K~1 >= K~
    for j, r in enumerate(rows):
        x = sub.row(j)
        L = x.size
        # the pipeline's selection equals the plain definition as a set
        assert np.array_equal(np.sort(oi[j]), np.sort(pi[j])), (wl.name, r)
        assert np.array_equal(np.sort(ov[j].view(np.uint32)), np.sort(pv[j].view(np.uint32)))
        t = tr[j]
        if L <= K:
            assert t[0] == oracle.ROUTE_DIRECT
            continue
        c = oracle.coarse(x).astype(np.int64)
        a = oracle.phase(j, s)
        view = np.arange(L)[np.arange(L) % s == a]
        assert t[1] == view.size  # |V| by direct count (eq:method:view)
        route = t[0] & ~oracle.ROUTE_REREAD_FLAG
        if t[2] >= 0:
            cv = np.sort(c[view])
            assert t[2] == cv[q0 - 1] and t[3] == cv[q1 - 1]  # order statistics
            assert t[4] == np.count_nonzero(c <= t[2])
            if t[4] >= K:  # containment lemma: the admitted tail holds a Top-K
                top = set(pi[j].tolist())
                assert top <= set(np.nonzero(c <= t[2])[0].tolist())
                assert route in (oracle.ROUTE_PRIMARY, oracle.ROUTE_EXACT_OVERFLOW)
            else:
                assert t[5] == np.count_nonzero(c <= t[3])
        else:
            assert route == oracle.ROUTE_EXACT_UNSAMPLED
            assert L < pol.l_samp_min or view.size < q1
        if route >= oracle.ROUTE_EXACT_UNSAMPLED:
            tstar = np.sort(c)[K - 1]
            assert t[6] == tstar
            assert t[7] == np.count_nonzero(c == tstar)
            assert bool(t[0] & oracle.ROUTE_REREAD_FLAG) == (t[7] > pol.cap)
        else:
            assert t[6] == -1
    return tr


def test_route_model_tiny_config():
    wl = W.tiny()
    _route_checks(wl, wl.K, oracle.default_policy(l_samp_min=0))


def test_route_model_decode_rows():
    wl = W.decode()
    tr = _route_checks(wl, wl.K, oracle.default_policy(), rows=range(0, 64, 4))
    assert np.all((tr[:, 0] == oracle.ROUTE_PRIMARY) | (tr[:, 0] == oracle.ROUTE_BAND)
                  | (tr[:, 0] == oracle.ROUTE_EXACT_UNDERFILL))


def test_route_model_adversarial_rows():
    wl = W.adversarial(n_rows=64)
    _route_checks(wl, wl.K, oracle.default_policy())
    wl = W.adversarial_recovery(n_rows=32)
    tr = _route_checks(wl, wl.K, oracle.default_policy())
    strided = tr[2::4]
    assert np.any(strided[:, 0] == oracle.ROUTE_EXACT_UNDERFILL)


@pytest.mark.parametrize("kind", ["clustered", "block"])
def test_route_model_tie_rows(kind):
    """Decode-shaped rows with heavy ties: a boundary bin over the frontier
    is resolved by re-reading (every "block" row, the longer "clustered"
    rows), and the exact route's invariants hold on a sample of rows."""
    wl = W.decode_ties(kind)
    _, _, tr = oracle.route_model(wl.scores, wl.row_offsets, wl.row_lengths, wl.K,
                                  oracle.default_policy())
    reread = (tr[:, 0] & oracle.ROUTE_REREAD_FLAG) != 0
    if kind == "block":
        assert reread.all()
    else:
        assert 0 < reread.sum() < wl.n_rows
        assert wl.row_lengths[reread].min() > wl.row_lengths[~reread].min()
    _route_checks(wl, wl.K, oracle.default_policy(), rows=range(0, 64, 8))


@pytest.mark.parametrize("s,cap,lmin", [(64, 8192, 0), (128, 600, 0), (256, 8192, 4096), (2, 50, 0)])
def test_route_model_policies(s, cap, lmin):
    rng = np.random.default_rng(s + cap)
    rows = []
    for L in (300, 999, 1000, 1001, 4096, 20000):
        x = rng.standard_normal(L).astype(np.float32)
        rows.append(x)
        rows.append(np.round(x * 4).astype(np.float32))       # heavy ties
        rows.append(np.full(L, 1.5, np.float32))              # all equal
    buf = np.concatenate(rows)
    lens = np.array([r.size for r in rows], np.int32)
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    wl = W.Workload("policies", buf, offs, lens, 1000, "")
    _route_checks(wl, 1000, oracle.default_policy(s=s, cap=cap, l_samp_min=lmin))


def test_route_model_nested_target_below_the_primary():
    """A policy whose nested target K~1 is below K~ (rho1 < rho) gets
    K~1 = K~: the nested boundary is never tighter than the primary one, so a
    row is sampled only when its view holds the primary rank, and tau1 =
    tau0.  Rows whose view size falls between the two ranks take the exact
    route.  (K = 1000, s = 4: q0 = 1250, the unraised q1 would be 375.)"""
    rng = np.random.default_rng(61)
    rows = []
    for L in (1600, 3000, 4999, 5000, 5001, 5003, 9000):
        x = rng.standard_normal(L).astype(np.float32)
        rows.append(x)
        rows.append(np.round(x * 4).astype(np.float32))
    buf = np.concatenate(rows)
    lens = np.array([r.size for r in rows], np.int32)
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    wl = W.Workload("nested below primary", buf, offs, lens, 1000, "")
    pol = oracle.default_policy(s=4, rho_num=5, rho_den=1, rho1_num=3, rho1_den=2, l_samp_min=0)
    tr = _route_checks(wl, 1000, pol)
    q0 = math.ceil(5 * 1000 / 4)
    for j in range(wl.n_rows):
        if tr[j][2] >= 0:
            assert tr[j][1] >= q0 and tr[j][3] == tr[j][2]
        elif lens[j] > 1000:
            assert tr[j][1] < q0 and tr[j][0] == oracle.ROUTE_EXACT_UNSAMPLED
    assert np.any(tr[:, 2] >= 0) and np.any((tr[:, 2] < 0) & (lens > 1000))
