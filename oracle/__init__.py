"""CPU oracle for exact Top-K over ragged FP32 rows.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``; the GPU library and its Python binding
never import it.  The arithmetic lives in ``topk_oracle.c`` (plain C, built by
``oracle.build``); this module only marshals numpy arrays.

Functions and the passages they follow:

* ``topk_ragged``  -- the plain definition of the operator (Section 2.1,
  operator contract; exactness criterion eq:eval:exactness), with the tie rule
  "lowest index wins" and -0.0 < +0.0 from the order-preserving uint32 key.
* ``route_model``  -- the sample-guided pipeline of Section 4 step by step
  (eq:method:view .. eq:method:refine-recurrence), reporting per row the route
  and the integers that decide it.
* ``asc32`` / ``fp16_rn`` / ``coarse`` / ``cutoffs`` -- the ordered key, the
  FP16 projection and coarse map (eq:method:coarse-map) and the inclusive FP32
  endpoint of each coarse bin (Section 4.3).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .build import LIB_PATH, build as _build

ROUTE_DIRECT = 0
ROUTE_PRIMARY = 1
ROUTE_BAND = 2
ROUTE_EXACT_UNSAMPLED = 3
ROUTE_EXACT_UNDERFILL = 4
ROUTE_EXACT_OVERFLOW = 5
ROUTE_REREAD_FLAG = 16
TRACE_WORDS = 8

_lib = None


class Policy(ctypes.Structure):
    """Sampled-pipeline policy (see ``oracle_policy`` in topk_oracle.c)."""

    _fields_ = [
        ("s", ctypes.c_int32),
        ("rho_num", ctypes.c_int32),
        ("rho_den", ctypes.c_int32),
        ("rho1_num", ctypes.c_int32),
        ("rho1_den", ctypes.c_int32),
        ("l_samp_min", ctypes.c_int32),
        ("cap", ctypes.c_int32),
    ]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            _build()
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        L.oracle_topk_ragged.argtypes = [P, P, P, ctypes.c_int32, ctypes.c_int32, P, P, ctypes.c_int]
        L.oracle_topk_ragged.restype = ctypes.c_int
        L.oracle_route_model.argtypes = [P, P, P, P, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.POINTER(Policy), P, P, P, ctypes.c_int]
        L.oracle_route_model.restype = ctypes.c_int
        L.oracle_asc32.argtypes = [ctypes.c_uint32]
        L.oracle_asc32.restype = ctypes.c_uint32
        L.oracle_coarse.argtypes = [ctypes.c_float]
        L.oracle_coarse.restype = ctypes.c_uint32
        L.oracle_fp16_rn.argtypes = [ctypes.c_float]
        L.oracle_fp16_rn.restype = ctypes.c_uint16
        L.oracle_cutoff.argtypes = [ctypes.c_uint32]
        L.oracle_cutoff.restype = ctypes.c_uint32
        L.oracle_phase.argtypes = [ctypes.c_int32, ctypes.c_int32]
        L.oracle_phase.restype = ctypes.c_int32
        L.oracle_sample_rank.argtypes = [ctypes.c_int32] * 4
        L.oracle_sample_rank.restype = ctypes.c_int32
        L.oracle_coarse_many.argtypes = [P, ctypes.c_int64, P]
        L.oracle_fp16_many.argtypes = [P, ctypes.c_int64, P]
        L.oracle_asc32_many.argtypes = [P, ctypes.c_int64, P]
        L.oracle_cutoff_all.argtypes = [P]
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def _rows(scores, row_offsets, row_lengths):
    scores = np.ascontiguousarray(scores, dtype=np.float32)
    offs = np.ascontiguousarray(row_offsets, dtype=np.int64)
    lens = np.ascontiguousarray(row_lengths, dtype=np.int32)
    assert offs.shape == lens.shape
    for r in range(len(lens)):  # rows must lie inside the score buffer
        L = max(0, int(lens[r]))
        assert 0 <= offs[r] and offs[r] + L <= scores.size, (r, offs[r], L)
    return scores, offs, lens


def topk_ragged(scores, row_offsets, row_lengths, K: int, n_threads: int = 0):
    """Plain-definition Top-K.  Returns (idx [n, K] int32, val [n, K] float32)."""
    scores, offs, lens = _rows(scores, row_offsets, row_lengths)
    n = len(lens)
    oi = np.empty((n, K), np.int32)
    ov = np.empty((n, K), np.float32)
    rc = lib().oracle_topk_ragged(_ptr(scores), _ptr(offs), _ptr(lens), n, K,
                                  _ptr(oi), _ptr(ov), n_threads)
    if rc != 0:
        raise RuntimeError(f"oracle_topk_ragged failed: {rc}")
    return oi, ov


def default_policy(**kw) -> Policy:
    """The pipeline constants of the evaluated configuration: s = 128,
    K~ = 1.5 K, K~1 = 1.75 K (Sections 4.2 and 6.4), plus the sampling floor
    and frontier capacity of this implementation."""
    p = dict(s=128, rho_num=3, rho_den=2, rho1_num=7, rho1_den=4, l_samp_min=8192, cap=6144)
    p.update(kw)
    return Policy(**p)


def route_model(scores, row_offsets, row_lengths, K: int, policy: Policy | None = None,
                n_threads: int = 0, row_ids=None):
    """Step-by-step pipeline model.  Returns (idx, val, trace [n, 8] int32).
    row_ids: original row numbers (they select the view phase) when the rows
    are a subset of a larger call."""
    scores, offs, lens = _rows(scores, row_offsets, row_lengths)
    policy = policy or default_policy()
    n = len(lens)
    ids = None
    if row_ids is not None:
        ids = np.ascontiguousarray(row_ids, dtype=np.int32)
        assert ids.shape == lens.shape
    oi = np.empty((n, K), np.int32)
    ov = np.empty((n, K), np.float32)
    tr = np.empty((n, TRACE_WORDS), np.int32)
    rc = lib().oracle_route_model(_ptr(scores), _ptr(offs), _ptr(lens),
                                  _ptr(ids) if ids is not None else None, n, K,
                                  ctypes.byref(policy), _ptr(oi), _ptr(ov), _ptr(tr), n_threads)
    if rc != 0:
        raise RuntimeError(f"oracle_route_model failed: {rc}")
    return oi, ov, tr


def asc32(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint32)
    out = np.empty_like(b)
    lib().oracle_asc32_many(_ptr(b), b.size, _ptr(out))
    return out


def fp16_rn(x: np.ndarray) -> np.ndarray:
    """FP16 bit patterns (uint16) of round-to-nearest-even projection."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().oracle_fp16_many(_ptr(x), x.size, _ptr(out))
    return out


def coarse(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.uint32)
    lib().oracle_coarse_many(_ptr(x), x.size, _ptr(out))
    return out


def cutoffs() -> np.ndarray:
    """Inclusive ascending-key endpoint of every coarse bin, uint32[2048]."""
    out = np.empty(2048, np.uint32)
    lib().oracle_cutoff_all(_ptr(out))
    return out


def phase(r: int, s: int) -> int:
    return lib().oracle_phase(r, s)


def sample_rank(K: int, num: int, den: int, s: int) -> int:
    return lib().oracle_sample_rank(K, num, den, s)
