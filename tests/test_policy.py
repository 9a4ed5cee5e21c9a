"""The per-K policy (topk_ragged_policy_for_k) against the exchangeable model
of the view (eq:insight:exchangeable): under positional exchangeability the
complete-row rank J(q) of the q-th largest of the n_a = floor(L / s) view
samples is a finite-population order statistic, J(q) - q being negative
hypergeometric (the unsampled elements met before the q-th sampled one when
the row is scanned from its largest value down).  An underfilled proposal
needs C(tau) < K, and C(tau) >= J(q) (the boundary bin holds the q-th sample
and everything above it), so P(J(q) < K) bounds the underfill rate; the
frontier overflows when C(tau0) exceeds the capacity, which J(q0) > cap
tracks for continuous scores.  The recalibrated constants must keep the
nested boundary's underfill rate within that of the evaluated configuration
at K = 2048, and the primary overflow rate below 1 %.  Host-only: no GPU."""
import numpy as np
import pytest
from scipy.stats import nhypergeom

CAP = 6144
INT32_MAX = 2**31 - 1


@pytest.fixture(scope="module")
def topk():
    import torch  # noqa: F401

    from paper_2609_08450_amd import topk as T
    T.lib()
    return T


def sample_rank(K, num, den, s):
    return -(-num * K // (den * s))


def p_underfill(L, s, q, K):
    n = L // s
    return float(nhypergeom(L, L - n, q).cdf(K - q - 1)) if K - q - 1 >= 0 else 0.0


def p_overflow(L, s, q, cap):
    n = L // s
    return float(nhypergeom(L, L - n, q).sf(cap - q))


def ranks(p, K):
    s = 1 << p.s_log2
    return s, sample_rank(K, p.rho_num, p.rho_den, s), sample_rank(K, p.rho1_num, p.rho1_den, s)


def test_evaluated_configuration_is_kept_at_k2048(topk):
    assert topk.policy_for_k(2048).as_dict() == topk.default_policy().as_dict()
    assert topk.policy_for_k(2559).as_dict() == topk.default_policy().as_dict()


def test_model_reproduces_a_textbook_case():
    # s = 1 (every element sampled): J(q) = q exactly
    assert p_underfill(1000, 1, 10, 11) == 1.0 and p_underfill(1000, 1, 10, 10) == 0.0
    # mean of the order statistic: q (L + 1) / (n + 1)
    L, s, q = 4096, 16, 5
    n = L // s
    X = nhypergeom(L, L - n, q)
    assert abs(X.mean() + q - q * (L + 1) / (n + 1)) < 1e-9
    # and its variance, q (n - q + 1) (L + 1) (L - n) / ((n + 1)^2 (n + 2))
    var = q * (n - q + 1) * (L + 1) * (L - n) / ((n + 1) ** 2 * (n + 2))
    assert abs(X.var() - var) < 1e-6 * var


@pytest.mark.parametrize("K", [1, 2, 17, 64, 200, 256, 383, 384, 512, 767, 768, 1024, 1535,
                               1536, 2047, 2048, 2559, 2560, 3072, 4096, 4351])
def test_per_k_constants_keep_the_evaluated_risk(topk, K):
    ref = topk.default_policy()
    s0, _, q1_ref = ranks(ref, 2048)
    p = topk.policy_for_k(K)
    assert p.l_samp_min == (8192 if K < 2048 else -4) and p.cap == CAP
    s, q0, q1 = ranks(p, K)
    assert 1 <= q0 <= q1
    assert q0 * s >= K                      # the proposal targets at least K
    floor = 8192 if K < 2048 else 4 * K
    for L in (max(floor, q1 * s), 65536, 131072):
        if L // s < q1:
            continue                        # the row would take the exact route
        ref_under = p_underfill(L, s0, q1_ref, 2048) if L >= 8192 else p_underfill(8192, s0, q1_ref, 2048)
        assert p_underfill(L, s, q1, K) <= ref_under * 1.05, (K, L)
        assert p_overflow(L, s, q0, CAP) <= 0.01, (K, L)


@pytest.mark.parametrize("K", [4352, 5000, 8192, 16384])
def test_large_k_takes_the_exact_route(topk, K):
    assert topk.policy_for_k(K).l_samp_min == INT32_MAX


def test_policy_for_k_argument_checks(topk):
    import ctypes

    L = topk.lib()
    p = topk.Policy()
    assert L.topk_ragged_policy_for_k(0, ctypes.byref(p)) == -1
    assert L.topk_ragged_policy_for_k(16385, ctypes.byref(p)) == -1
    assert L.topk_ragged_policy_for_k(2048, None) == -1
