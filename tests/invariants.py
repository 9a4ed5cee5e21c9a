"""Exactness checks for one row, written independently of the oracle.

The selected set must be the first min(K, L) positions of the row ranked by
(value descending, +0.0 before -0.0, index ascending) -- computed here with
numpy's lexsort -- and every returned value must be the bit-exact score.
"""
from __future__ import annotations

import numpy as np

NEG_INF_BITS = np.float32(-np.inf).view(np.uint32)


def reference_rank(x: np.ndarray) -> np.ndarray:
    """Positions of x in selection order, via numpy lexsort on numeric value."""
    x = np.asarray(x, np.float32)
    idx = np.arange(x.size)
    neg = -x.astype(np.float64)
    sign = np.signbit(x).astype(np.int8)  # -0.0 ranks after +0.0
    return np.lexsort((idx, sign, neg))


def check_row(x: np.ndarray, K: int, out_idx: np.ndarray, out_val: np.ndarray, where: str = ""):
    x = np.asarray(x, np.float32)
    L = x.size
    oi = np.asarray(out_idx, np.int64)
    ov = np.asarray(out_val, np.float32).view(np.uint32)
    assert oi.shape == (K,) and ov.shape == (K,), where
    if L <= K:
        exp = np.full(K, -1, np.int64)
        exp[:L] = np.arange(L)
        assert np.array_equal(oi, exp), f"{where}: direct layout wrong"
        ev = np.full(K, NEG_INF_BITS, np.uint32)
        ev[:L] = x.view(np.uint32)
        assert np.array_equal(ov, ev), f"{where}: direct values wrong"
        return
    assert oi.min() >= 0 and oi.max() < L, f"{where}: index out of range"
    assert np.unique(oi).size == K, f"{where}: duplicate indices"
    assert np.array_equal(ov, x.view(np.uint32)[oi]), f"{where}: value bits differ from scores"
    want = np.sort(reference_rank(x)[:K])
    got = np.sort(oi)
    assert np.array_equal(got, want), f"{where}: selected set differs from the exact Top-K"


def canonical(out_idx: np.ndarray, out_val: np.ndarray):
    """Per-row (index, value-bits) pairs sorted by index, for set comparison."""
    oi = np.asarray(out_idx, np.int64)
    ov = np.asarray(out_val, np.float32).view(np.uint32).astype(np.int64)
    order = np.argsort(oi, axis=-1, kind="stable")
    return np.take_along_axis(oi, order, -1), np.take_along_axis(ov, order, -1)
