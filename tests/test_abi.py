"""CPU checks of the C-ABI library: it loads, exports every function the
header declares, and rejects bad arguments on the host (no GPU needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "topk_ragged.h")


@pytest.fixture(scope="module")
def lib():
    import torch  # noqa: F401  (binds the library to torch's HIP runtime)

    from paper_2609_08450_amd import topk
    from paper_2609_08450_amd.build import LIB_PATH

    if not os.path.exists(LIB_PATH):
        pytest.fail("libtopk_ragged.so is not built (run __graft_entry__.build())")
    return topk.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(topk_ragged\w*)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for must in ("topk_ragged", "topk_ragged_ex", "topk_ragged_workspace_size",
                 "topk_ragged_workspace_init", "topk_ragged_read_stats"):
        assert must in names


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_host_argument_checks(lib):
    P = ctypes.c_void_p
    n = None
    assert lib.topk_ragged(n, n, n, 0, 2048, n, n, n, n) == 0              # no rows: no-op
    assert lib.topk_ragged(n, n, n, -1, 2048, n, n, n, n) == -1
    assert lib.topk_ragged(n, n, n, 4, 0, n, n, n, n) == -1
    assert lib.topk_ragged(n, n, n, 4, 16385, n, n, n, n) == -1
    assert lib.topk_ragged(n, n, n, 4, 2048, n, n, n, n) == -1             # null pointers
    dummy = P(16)
    bad = lib.Policy if hasattr(lib, "Policy") else None
    assert lib.topk_ragged_workspace_size(-1, 2048) == 0
    assert lib.topk_ragged_workspace_size(4, 0) == 0
    assert lib.topk_ragged_workspace_init(n, 0, 4, 2048, n) == -1
    # a workspace that is not 256-byte aligned is refused before any device work
    assert lib.topk_ragged_workspace_init(P(4096 + 8), 1 << 20, 4, 2048, n) == -1
    assert lib.topk_ragged(P(16), P(16), P(16), 4, 2048, P(16), P(16), P(4096 + 8), n) == -1
    from paper_2609_08450_amd.topk import Stats
    assert lib.topk_ragged_read_stats(P(4096 + 8), ctypes.byref(Stats()), n) == -1
    assert lib.topk_ragged_read_stats(n, n, n) == -1
    assert lib.topk_ragged_debug_cutoffs(n, n) == -1
    assert lib.topk_ragged_debug_coarse(n, -1, n, n) == -1
    assert lib.topk_ragged_debug_coarse(n, 0, n, n) == 0
    assert lib.topk_ragged_status_str(-1) == b"invalid argument"
    # the allocation-free call: its row limit and scalar checks come first
    assert lib.topk_ragged_noalloc(n, n, n, 16385, 2048, n, n, n) == -4
    assert lib.topk_ragged_noalloc(n, n, n, 0, 2048, n, n, n) == 0
    assert lib.topk_ragged_noalloc(n, n, n, -1, 2048, n, n, n) == -1
    assert lib.topk_ragged_noalloc(n, n, n, 4, 0, n, n, n) == -1
    assert lib.topk_ragged_noalloc(n, n, n, 4, 2048, n, n, n) == -1       # null pointers
    del dummy, bad


def test_policy_checks(lib):
    from paper_2609_08450_amd import topk

    pol = topk.default_policy()
    P = ctypes.c_void_p(16)
    for field, value in (("s_log2", 13), ("s_log2", -1), ("cap", 0), ("cap", 6145),
                         ("rho_den", 0), ("rho1_num", 0)):
        p = topk.default_policy()
        setattr(p, field, value)
        rc = lib.topk_ragged_ex(P, P, P, 4, 2048, P, P, P, ctypes.byref(p), None, None)
        assert rc == -1, (field, value)
    del pol


def test_default_policy_is_the_evaluated_configuration(lib):
    from paper_2609_08450_amd import topk

    p = topk.default_policy().as_dict()
    assert p["s_log2"] == 7                        # s = 128
    assert (p["rho_num"], p["rho_den"]) == (3, 2)  # K~ = 1.5 K
    assert (p["rho1_num"], p["rho1_den"]) == (7, 4)  # K~1 = 1.75 K
    assert p["cap"] == topk.FRONTIER_CAP


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    from paper_2609_08450_amd import topk

    monkeypatch.setattr(topk, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(topk, "_lib", None)
    with pytest.raises(topk.TopkError):
        topk.lib()
