"""Seeded synthetic score rows shaped like the paper's workloads.

This module holds only input generation: no selection arithmetic.  Both the GPU
parity tests and the CPU oracle consume its arrays.  The paper measures on
indexer-score captures of a production model and on framework traces, which
are not available; these generators stand in for them with the structure the
paper describes (Section 3 observations: heavy upper tail near the row end,
runs of relevant tokens; eq:indexer for the chunked-prefill block).

Every workload is deterministic in its seed: row lengths are drawn first from
the parent PCG64 stream, then each row draws from its own child stream
(``SeedSequence.spawn``), so any single row can be regenerated alone.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

BASE_SEED = 260908450
VIEW_STRIDE = 128  # stride of the sampled view, used by the strided-adversary rows


@dataclasses.dataclass
class Workload:
    name: str
    scores: np.ndarray       # float32, 1-D buffer holding every row
    row_offsets: np.ndarray  # int64 [n_rows], element offset of row r
    row_lengths: np.ndarray  # int32 [n_rows], valid length of row r
    K: int
    description: str

    @property
    def n_rows(self) -> int:
        return int(self.row_lengths.size)

    @property
    def total_len(self) -> int:
        return int(np.maximum(self.row_lengths, 0).astype(np.int64).sum())

    def row(self, r: int) -> np.ndarray:
        o, L = int(self.row_offsets[r]), max(0, int(self.row_lengths[r]))
        return self.scores[o:o + L]

    def subset(self, rows) -> "Workload":
        """Workload made of the given rows only, packed contiguously."""
        rows = list(rows)
        parts = [self.row(r) for r in rows]
        lens = np.array([p.size for p in parts], np.int32)
        offs = np.zeros(len(rows), np.int64)
        if len(rows) > 1:
            offs[1:] = np.cumsum(lens[:-1], dtype=np.int64)
        buf = np.concatenate(parts) if parts else np.zeros(0, np.float32)
        return Workload(f"{self.name}[subset]", buf.astype(np.float32, copy=False), offs, lens,
                        self.K, self.description)


def _pack(rows: list[np.ndarray]):
    lens = np.array([r.size for r in rows], np.int32)
    offs = np.zeros(len(rows), np.int64)
    if len(rows) > 1:
        offs[1:] = np.cumsum(lens[:-1], dtype=np.int64)
    buf = np.concatenate(rows).astype(np.float32, copy=False) if rows else np.zeros(0, np.float32)
    return buf, offs, lens


def _children(seed: int, n: int):
    ss = np.random.SeedSequence(seed)
    parent = np.random.Generator(np.random.PCG64(ss))
    kids = [np.random.Generator(np.random.PCG64(c)) for c in ss.spawn(n)]
    return parent, kids


def decode_mixture_row(rng: np.random.Generator, L: int) -> np.ndarray:
    """Indexer-like decode row: N(0,1) base, a recency bump 0.5*exp(-(L-1-j)/4096)
    toward the row end, and 1% of positions in runs of 64 consecutive tokens
    (distinct 64-aligned blocks) replaced by N(3, 0.5)."""
    x = rng.standard_normal(L, dtype=np.float32)
    j = np.arange(L, dtype=np.float64)
    x += (0.5 * np.exp(-(L - 1 - j) / 4096.0)).astype(np.float32)
    nblocks = L // 64
    n_runs = min(nblocks, int(round(0.01 * L / 64)))
    if n_runs > 0:
        blocks = rng.choice(nblocks, size=n_runs, replace=False)
        for b in blocks:
            x[b * 64:(b + 1) * 64] = rng.normal(3.0, 0.5, 64).astype(np.float32)
    return x


def tiny(seed: int = BASE_SEED + 1) -> Workload:
    """4 rows, L uniform in [1024, 8192], K = 256, i.i.d. N(0,1)."""
    parent, kids = _children(seed, 4)
    lens = parent.integers(1024, 8192, size=4, endpoint=True)
    rows = [kids[r].standard_normal(int(lens[r]), dtype=np.float32) for r in range(4)]
    buf, offs, ls = _pack(rows)
    return Workload("tiny", buf, offs, ls, 256, "4 rows, L~U[1024,8192], K=256, N(0,1)")


def decode(seed: int = BASE_SEED + 2, n_rows: int = 64) -> Workload:
    """64 rows, L uniform in [16384, 131072], K = 2048, decode mixture."""
    parent, kids = _children(seed, n_rows)
    lens = parent.integers(16384, 131072, size=n_rows, endpoint=True)
    rows = [decode_mixture_row(kids[r], int(lens[r])) for r in range(n_rows)]
    buf, offs, ls = _pack(rows)
    return Workload("decode", buf, offs, ls, 2048,
                    f"{n_rows} rows, L~U[16384,131072], K=2048, decode mixture")


def chunked_prefill(seed: int = BASE_SEED + 3, n_rows: int = 4096, context: int = 131072,
                    dim: int = 64, heads: int = 8, K: int = 2048) -> Workload:
    """Causal prefill block over one context: row i has valid length
    context - n_rows + 1 + i and pitch `context`.  Scores follow eq:indexer:
    s_ij = sum_h w_h * relu(q_ih . k_j / sqrt(dim)), keys and head weights
    shared by all rows, all FP32."""
    ss = np.random.SeedSequence(seed)
    g = np.random.Generator(np.random.PCG64(ss))
    keys = g.standard_normal((context, dim), dtype=np.float32)
    w = g.random(heads, dtype=np.float32)
    q = g.standard_normal((n_rows, heads, dim), dtype=np.float32)
    scale = np.float32(1.0 / math.sqrt(dim))
    out = np.empty((n_rows, context), np.float32)
    kt = np.ascontiguousarray(keys.T)
    chunk = 32
    for r0 in range(0, n_rows, chunk):
        r1 = min(n_rows, r0 + chunk)
        acc = np.zeros((r1 - r0, context), np.float32)
        for h in range(heads):
            d = q[r0:r1, h, :] @ kt
            d *= scale
            np.maximum(d, 0, out=d)
            d *= w[h]
            acc += d
        out[r0:r1] = acc
    lens = (context - n_rows + 1 + np.arange(n_rows)).astype(np.int32)
    offs = (np.arange(n_rows, dtype=np.int64) * context)
    return Workload("chunked_prefill", out.reshape(-1), offs, lens, K,
                    f"{n_rows} causal rows over a {context}-token context, pitch {context}, "
                    f"indexer scores (dim {dim}, {heads} heads), K={K}")


def long_split(seed: int = BASE_SEED + 4, n_rows: int = 16) -> Workload:
    """16 rows, L uniform in [524288, 1048576], K = 2048, decode mixture."""
    parent, kids = _children(seed, n_rows)
    lens = parent.integers(524288, 1048576, size=n_rows, endpoint=True)
    rows = [decode_mixture_row(kids[r], int(lens[r])) for r in range(n_rows)]
    buf, offs, ls = _pack(rows)
    return Workload("long_split", buf, offs, ls, 2048,
                    f"{n_rows} rows, L~U[524288,1048576], K=2048, decode mixture")


def view_phase(r: int, s: int = VIEW_STRIDE) -> int:
    """Residue class read by the sampled view of row r: bit reversal of
    (r mod s) over log2(s) bits.  Needed here only to place the strided
    adversary's values on that residue class."""
    nb = s.bit_length() - 1
    v = r % s
    return int(format(v, f"0{nb}b")[::-1], 2) if nb > 0 else 0


def adversarial(seed: int = BASE_SEED + 5, n_rows: int = 1024, K: int = 2048,
                onstride_mean: float = -2.0, onstride_sd: float = 1.0) -> Workload:
    """Edge mix, case = r mod 4:
    (a) L log-uniform in [512, K-1], N(0,1)            (direct path, -1 padding)
    (b) per-row codebook of 256 distinct N(0,1) values (heavy ties)
    (c) view residue N(onstride_mean, onstride_sd), elsewhere N(0,1)
    (d) each entry -inf with probability 0.3, else N(0,1)
    (b)-(d) have L log-uniform in [512, 262144]."""
    parent, kids = _children(seed, n_rows)
    u = parent.random(n_rows)
    rows = []
    for r in range(n_rows):
        case = r % 4
        hi = (K - 1) if case == 0 else 262144
        L = int(math.floor(math.exp(math.log(512) + u[r] * (math.log(hi) - math.log(512)))))
        L = max(512, min(hi, L))
        g = kids[r]
        if case == 0:
            x = g.standard_normal(L, dtype=np.float32)
        elif case == 1:
            book = np.unique(g.standard_normal(4096, dtype=np.float32))
            book = g.permutation(book)[:256]
            x = book[g.integers(0, book.size, L)]
        elif case == 2:
            x = g.standard_normal(L, dtype=np.float32)
            a = view_phase(r)
            m = (L - a + VIEW_STRIDE - 1) // VIEW_STRIDE if a < L else 0
            x[a::VIEW_STRIDE] = g.normal(onstride_mean, onstride_sd, m).astype(np.float32)
        else:
            x = g.standard_normal(L, dtype=np.float32)
            x[g.random(L) < 0.3] = -np.inf
        rows.append(x.astype(np.float32, copy=False))
    buf, offs, ls = _pack(rows)
    return Workload("adversarial", buf, offs, ls, K,
                    f"{n_rows} rows, four edge cases (direct, ties, strided adversary "
                    f"N({onstride_mean},{onstride_sd}), 30% -inf), K={K}")


def decode_ties(kind: str, seed: int = BASE_SEED + 7, K: int = 2048) -> Workload:
    """Decode-shaped rows (the decode batch's lengths) with heavy ties:
    kind "clustered": each row drawn from its own codebook, the lowest 256 of
    4096 N(0,1) draws (so about a dozen codebook values share a coarse bin,
    and the boundary bin of the longer rows holds more than the frontier);
    kind "block": the decode mixture rows with 8000 random positions set to
    one value just above the row's K-th largest score."""
    base = decode()
    g = np.random.default_rng(seed)
    rows = []
    for r in range(base.n_rows):
        L = int(base.row_lengths[r])
        if kind == "clustered":
            book = np.unique(g.standard_normal(4096, dtype=np.float32))[:256]
            x = book[g.integers(0, book.size, L)]
        elif kind == "block":
            x = base.row(r).copy()
            x[g.choice(L, 8000, replace=False)] = np.partition(x, L - K)[L - K] + np.float32(0.01)
        else:
            raise ValueError(kind)
        rows.append(x.astype(np.float32, copy=False))
    buf, offs, ls = _pack(rows)
    return Workload(f"decode ties ({kind})", buf, offs, ls, K,
                    f"decode lengths, heavy ties ({kind}), K={K}")


def adversarial_recovery(seed: int = BASE_SEED + 6, n_rows: int = 256) -> Workload:
    """Variant of the edge mix whose strided rows carry N(3, 0.5) on the view
    residue: the view then sees only high values, the proposal underfills and
    the rows take the band and exact recovery routes."""
    w = adversarial(seed, n_rows, onstride_mean=3.0, onstride_sd=0.5)
    w.name = "adversarial_recovery"
    return w


CONFIGS = {
    1: tiny,
    2: decode,
    3: chunked_prefill,
    4: long_split,
    5: adversarial,
}


def make(config: int, **kw) -> Workload:
    return CONFIGS[config](**kw)


def chunked_prefill_device(device, seed: int = BASE_SEED + 3, n_rows: int = 4096,
                           context: int = 131072, dim: int = 64, heads: int = 8, K: int = 2048):
    """The chunked-prefill block with the indexer product computed on `device`
    (torch, FP32): the same seeded queries, keys and head weights as
    `chunked_prefill`, much faster to build at full size.  Returns
    (scores [n_rows * context] device tensor, row_offsets, row_lengths) with
    numpy offsets/lengths; the score bits may differ from the host build."""
    import torch

    ss = np.random.SeedSequence(seed)
    g = np.random.Generator(np.random.PCG64(ss))
    keys = torch.from_numpy(g.standard_normal((context, dim), dtype=np.float32)).to(device)
    w = g.random(heads, dtype=np.float32)
    q = torch.from_numpy(g.standard_normal((n_rows, heads, dim), dtype=np.float32)).to(device)
    scale = 1.0 / math.sqrt(dim)
    out = torch.empty((n_rows, context), dtype=torch.float32, device=device)
    kt = keys.t().contiguous()
    chunk = 256
    for r0 in range(0, n_rows, chunk):
        r1 = min(n_rows, r0 + chunk)
        acc = torch.zeros((r1 - r0, context), dtype=torch.float32, device=device)
        for h in range(heads):
            d = torch.mm(q[r0:r1, h, :].contiguous(), kt)
            d.mul_(scale).clamp_(min=0).mul_(float(w[h]))
            acc.add_(d)
        out[r0:r1] = acc
    lens = (context - n_rows + 1 + np.arange(n_rows)).astype(np.int32)
    offs = np.arange(n_rows, dtype=np.int64) * context
    return out.reshape(-1), offs, lens
