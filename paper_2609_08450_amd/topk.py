"""Python binding of the topk_ragged C-ABI (argument marshalling only).

Every function here forwards device pointers of torch tensors and the stream
handle to libtopk_ragged.so; all selection work runs in its HIP kernels.  The
library must be built (``paper_2609_08450_amd.build``); there is no fallback.
torch is imported first so the library binds to the HIP runtime torch already
loaded (one runtime per process, shared streams and allocations).
"""
from __future__ import annotations

import ctypes
import os

import torch

from .build import LIB_PATH

TRACE_WORDS = 8
K_MAX = 16384
FRONTIER_CAP = 6144
ROUTE_NAMES = ["direct", "primary", "band", "exact_unsampled", "exact_underfill", "exact_overflow"]


class TopkError(RuntimeError):
    pass


class Policy(ctypes.Structure):
    """Mirror of topk_ragged_policy (include/topk_ragged.h)."""

    _fields_ = [
        ("s_log2", ctypes.c_int32),
        ("rho_num", ctypes.c_int32),
        ("rho_den", ctypes.c_int32),
        ("rho1_num", ctypes.c_int32),
        ("rho1_den", ctypes.c_int32),
        ("l_samp_min", ctypes.c_int32),
        ("cap", ctypes.c_int32),
    ]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class Stats(ctypes.Structure):
    """Mirror of topk_ragged_stats."""

    _fields_ = [
        ("route", ctypes.c_uint64 * 6),
        ("reread", ctypes.c_uint64),
        ("wait_fallback", ctypes.c_uint64),
        ("errors", ctypes.c_uint64),
    ]

    def as_dict(self):
        d = {n: int(self.route[i]) for i, n in enumerate(ROUTE_NAMES)}
        d.update(reread=int(self.reread), wait_fallback=int(self.wait_fallback),
                 errors=int(self.errors))
        return d


_lib = None


def _check_single_hip_runtime():
    paths = set()
    with open("/proc/self/maps") as fh:
        for ln in fh:
            if "libamdhip64" in ln:
                paths.add(os.path.realpath(ln.split()[-1]))
    if len(paths) > 1:
        raise TopkError(f"more than one HIP runtime is loaded: {sorted(paths)}")


def lib():
    """Loads libtopk_ragged.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise TopkError(f"{LIB_PATH} is missing: build it with "
                            "`python -m paper_2609_08450_amd.build` (no CPU fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        _check_single_hip_runtime()
        P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.topk_ragged.argtypes = [P, P, P, i32, i32, P, P, P, P]
        L.topk_ragged.restype = ctypes.c_int
        L.topk_ragged_ex.argtypes = [P, P, P, i32, i32, P, P, P, ctypes.POINTER(Policy), P, P]
        L.topk_ragged_ex.restype = ctypes.c_int
        L.topk_ragged_noalloc.argtypes = [P, P, P, i32, i32, P, P, P]
        L.topk_ragged_noalloc.restype = ctypes.c_int
        L.topk_ragged_workspace_size.argtypes = [i32, i32]
        L.topk_ragged_workspace_size.restype = ctypes.c_size_t
        L.topk_ragged_workspace_init.argtypes = [P, ctypes.c_size_t, i32, i32, P]
        L.topk_ragged_workspace_init.restype = ctypes.c_int
        L.topk_ragged_read_stats.argtypes = [P, ctypes.POINTER(Stats), P]
        L.topk_ragged_read_stats.restype = ctypes.c_int
        L.topk_ragged_default_policy.argtypes = [ctypes.POINTER(Policy)]
        L.topk_ragged_default_policy.restype = ctypes.c_int
        L.topk_ragged_policy_for_k.argtypes = [ctypes.c_int32, ctypes.POINTER(Policy)]
        L.topk_ragged_policy_for_k.restype = ctypes.c_int
        L.topk_ragged_debug_coarse.argtypes = [P, i64, P, P]
        L.topk_ragged_debug_coarse.restype = ctypes.c_int
        L.topk_ragged_debug_read_ceiling.argtypes = [P, P, P, i32, i32, P, P, P]
        L.topk_ragged_debug_read_ceiling.restype = ctypes.c_int
        L.topk_ragged_debug_cutoffs.argtypes = [P, P]
        L.topk_ragged_debug_cutoffs.restype = ctypes.c_int
        L.topk_ragged_debug_set_spin_limit.argtypes = [ctypes.c_int32]
        L.topk_ragged_debug_set_spin_limit.restype = ctypes.c_int
        L.topk_ragged_status_str.argtypes = [ctypes.c_int]
        L.topk_ragged_status_str.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(rc: int, what: str):
    if rc != 0:
        msg = lib().topk_ragged_status_str(rc).decode()
        raise TopkError(f"{what} failed: {msg} ({rc})")


def _ptr(t: torch.Tensor | None, dtype=None, name=""):
    if t is None:
        return None
    if not t.is_cuda:
        raise TopkError(f"{name} must be a device tensor")
    if dtype is not None and t.dtype != dtype:
        raise TopkError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise TopkError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def default_policy() -> Policy:
    """The evaluated configuration (the policy for K around 2048)."""
    p = Policy()
    _check(lib().topk_ragged_default_policy(ctypes.byref(p)), "topk_ragged_default_policy")
    return p


def policy_for_k(K: int) -> Policy:
    """The policy a call with this K uses when none is given."""
    p = Policy()
    _check(lib().topk_ragged_policy_for_k(K, ctypes.byref(p)), "topk_ragged_policy_for_k")
    return p


def workspace_size(max_rows: int, K: int) -> int:
    n = lib().topk_ragged_workspace_size(max_rows, K)
    if n == 0:
        raise TopkError("topk_ragged_workspace_size: invalid arguments or device")
    return int(n)


def workspace_init(workspace: torch.Tensor, max_rows: int, K: int, stream=None) -> None:
    _check(lib().topk_ragged_workspace_init(_ptr(workspace, torch.uint8, "workspace"),
                                            workspace.numel(), max_rows, K, _stream(stream)),
           "topk_ragged_workspace_init")


def alloc_workspace(max_rows: int, K: int, device="cuda", stream=None) -> torch.Tensor:
    """Allocates (through torch) and initialises a workspace."""
    ws = torch.empty(workspace_size(max_rows, K), dtype=torch.uint8, device=device)
    workspace_init(ws, max_rows, K, stream)
    return ws


def topk_ragged(scores, row_offsets, row_lengths, n_rows: int, K: int, out_idx, out_val,
                workspace, stream=None) -> None:
    """Forwards to topk_ragged(); see include/topk_ragged.h for the contract."""
    _check(lib().topk_ragged(_ptr(scores, torch.float32, "scores"),
                             _ptr(row_offsets, torch.int64, "row_offsets"),
                             _ptr(row_lengths, torch.int32, "row_lengths"), n_rows, K,
                             _ptr(out_idx, torch.int32, "out_idx"),
                             _ptr(out_val, torch.float32, "out_val"),
                             _ptr(workspace, torch.uint8, "workspace"), _stream(stream)),
           "topk_ragged")


def topk_ragged_ex(scores, row_offsets, row_lengths, n_rows: int, K: int, out_idx, out_val,
                   workspace, policy: Policy | None = None, row_trace=None, stream=None) -> None:
    """Forwards to topk_ragged_ex() (explicit policy, optional per-row trace)."""
    _check(lib().topk_ragged_ex(_ptr(scores, torch.float32, "scores"),
                                _ptr(row_offsets, torch.int64, "row_offsets"),
                                _ptr(row_lengths, torch.int32, "row_lengths"), n_rows, K,
                                _ptr(out_idx, torch.int32, "out_idx"),
                                _ptr(out_val, torch.float32, "out_val"),
                                _ptr(workspace, torch.uint8, "workspace"),
                                ctypes.byref(policy) if policy is not None else None,
                                _ptr(row_trace, torch.int32, "row_trace"), _stream(stream)),
           "topk_ragged_ex")


def topk_ragged_noalloc(scores, row_offsets, row_lengths, n_rows: int, K: int, out_idx, out_val,
                        stream=None) -> None:
    """Forwards to topk_ragged_noalloc() (the library's own workspace)."""
    _check(lib().topk_ragged_noalloc(_ptr(scores, torch.float32, "scores"),
                                     _ptr(row_offsets, torch.int64, "row_offsets"),
                                     _ptr(row_lengths, torch.int32, "row_lengths"), n_rows, K,
                                     _ptr(out_idx, torch.int32, "out_idx"),
                                     _ptr(out_val, torch.float32, "out_val"), _stream(stream)),
           "topk_ragged_noalloc")


def read_stats(workspace, stream=None) -> dict:
    st = Stats()
    _check(lib().topk_ragged_read_stats(_ptr(workspace, torch.uint8, "workspace"),
                                        ctypes.byref(st), _stream(stream)),
           "topk_ragged_read_stats")
    return st.as_dict()


def debug_coarse(x, out_c, stream=None) -> None:
    _check(lib().topk_ragged_debug_coarse(_ptr(x, torch.float32, "x"), x.numel(),
                                          _ptr(out_c, torch.int16, "out_c"), _stream(stream)),
           "topk_ragged_debug_coarse")


def debug_cutoffs(out_cut, stream=None) -> None:
    _check(lib().topk_ragged_debug_cutoffs(_ptr(out_cut, torch.int32, "out_cut"),
                                           _stream(stream)), "topk_ragged_debug_cutoffs")


def debug_read_ceiling(scores, row_offsets, row_lengths, n_rows: int, K: int, out_max,
                       workspace, stream=None) -> None:
    """Forwards to topk_ragged_debug_read_ceiling() (read-only ceiling of a
    call; out_max: int32 device tensor [n_rows], zeroed by the caller;
    workspace: an initialised workspace for at least n_rows rows)."""
    _check(lib().topk_ragged_debug_read_ceiling(_ptr(scores, torch.float32, "scores"),
                                                _ptr(row_offsets, torch.int64, "row_offsets"),
                                                _ptr(row_lengths, torch.int32, "row_lengths"),
                                                n_rows, K, _ptr(out_max, torch.int32, "out_max"),
                                                _ptr(workspace, torch.uint8, "workspace"),
                                                _stream(stream)),
           "topk_ragged_debug_read_ceiling")


def debug_set_spin_limit(polls: int) -> None:
    """Polls of the boundary word before a split segment builds the view
    itself, for later calls (0 = default); see include/topk_ragged.h."""
    _check(lib().topk_ragged_debug_set_spin_limit(polls), "topk_ragged_debug_set_spin_limit")


class TopK:
    """Convenience holder: a workspace sized for `max_rows` rows and rank K,
    plus output tensors; `__call__` forwards one topk_ragged call."""

    def __init__(self, max_rows: int, K: int, device="cuda"):
        self.max_rows, self.K = max_rows, K
        self.workspace = alloc_workspace(max_rows, K, device)

    def __call__(self, scores, row_offsets, row_lengths, out_idx=None, out_val=None,
                 policy: Policy | None = None, row_trace=None, stream=None):
        n = int(row_lengths.numel())
        if n > self.max_rows:
            raise TopkError(f"{n} rows exceed the workspace's {self.max_rows}")
        if out_idx is None:
            out_idx = torch.empty((n, self.K), dtype=torch.int32, device=scores.device)
        if out_val is None:
            out_val = torch.empty((n, self.K), dtype=torch.float32, device=scores.device)
        if policy is None and row_trace is None:
            topk_ragged(scores, row_offsets, row_lengths, n, self.K, out_idx, out_val,
                        self.workspace, stream)
        else:
            topk_ragged_ex(scores, row_offsets, row_lengths, n, self.K, out_idx, out_val,
                           self.workspace, policy, row_trace, stream)
        return out_idx, out_val
