"""The split-row segment plan's arithmetic, restated on the host.

The kernel cuts a row of length L into P segments of seg elements (a multiple
of 64) from target = max(kSegMin, ceil(total / items)) and P0 = min(pmax,
ceil(L / target)), with the two ceilings taken in FP64 and seg and P from an
FP64 floor division it treats as exact.  numpy's float64 division is IEEE
correctly rounded like the device's, so these checks hold for the kernel's
instructions too: the floor division is exact for 32-bit operands, and every
plan is valid (segments cover the row, none is empty, P <= pmax, and no
segment index reaches ceil(L / kSegMin), which the kernel's early exit
assumes).
"""
import numpy as np

K_SEG_MIN = 8192  # smallest segment target (kSegMin in the kernel)


def udiv32(x, y):
    return np.floor(np.float64(x) / np.float64(y)).astype(np.uint64)


def plan(L, total, items, pmax):
    tq = np.ceil(np.float64(total) / np.float64(items))
    target = np.uint64(max(float(K_SEG_MIN), min(float(tq), 2147483648.0)))
    P0 = min(pmax, int(np.ceil(np.float64(L) / np.float64(target))))
    seg = (int(udiv32(L + P0 - 1, P0)) + 63) & ~63
    P = int(udiv32(L + seg - 1, seg))
    return P0, seg, P


def test_fp64_floor_division_is_exact_for_32bit_operands():
    rng = np.random.default_rng(7)
    y = np.concatenate([np.arange(1, 2000, dtype=np.uint64),
                        rng.integers(1, 2**32, 20000, dtype=np.uint64),
                        (np.uint64(2**32) - np.arange(1, 2000, dtype=np.uint64))])
    # x = n y + (y - 1): the quotient is closest to the next integer
    n = (np.uint64(2**32 - 1) // y) - np.uint64(1)
    n = np.where(n > 0, rng.integers(0, 2**32, y.size, dtype=np.uint64) % (n + np.uint64(1)), 0)
    x = n * y + (y - np.uint64(1))
    keep = x < np.uint64(2**32)
    x, y = x[keep], y[keep]
    assert np.array_equal(udiv32(x, y), x // y)
    for xx in (2**32 - 1, 2**32 - 2, 2**31, 2**31 - 1):
        yy = np.arange(1, 5000, dtype=np.uint64)
        assert np.array_equal(udiv32(np.uint64(xx), yy), np.uint64(xx) // yy)


def test_plans_are_valid():
    rng = np.random.default_rng(11)
    Ls = np.concatenate([rng.integers(2049, 2**31, 3000), np.arange(2049, 40000, 7),
                         [K_SEG_MIN * k + d for k in range(1, 70) for d in (-1, 0, 1)]])
    for i, L in enumerate(Ls):
        L = int(L)
        if L < 2:
            continue
        pmax = int(2 ** rng.integers(1, 7))
        items = int(rng.integers(1, 2000))
        total = int(L + rng.integers(0, 2**40))
        if i % 5 == 0:
            total = L  # a lone row
        P0, seg, P = plan(L, total, items, pmax)
        assert 1 <= P <= P0 <= pmax
        assert seg % 64 == 0 and seg > 0
        assert (P - 1) * seg < L <= P * seg
        assert P <= -(-L // K_SEG_MIN)  # segment p < P has p * kSegMin < L


def _header_define(name):
    import os
    import re

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    text = open(os.path.join(root, "include", "topk_ragged.h")).read()
    return int(re.search(rf"#define {name} (0x[0-9A-Fa-f]+|\d+)", text).group(1), 0)


def _max_vector_byte_offset(off, beg, end, sh):
    """The row streaming's largest 16-byte vector offset from its base, the
    start of the 128-byte line holding element beg: the first vector is
    floor((off + beg + sh) / 4) rounded down to a multiple of 8, nvec =
    ceil((off + end + sh) / 4) - that, the last at byte (nvec - 1) * 16 (sh =
    the buffer's misalignment in elements, 0..3)."""
    v0 = ((off + beg + sh) >> 2) & ~7
    nvec = ((off + end + sh + 3) >> 2) - v0
    return (nvec - 1) * 16


def test_longest_row_keeps_32_bit_vector_offsets():
    """Rows of up to TOPK_L_MAX elements address every vector of any range of
    the row with a 32-bit byte offset, for every alignment of the buffer and
    the row; the first length past a few more elements would wrap."""
    lmax = _header_define("TOPK_L_MAX")
    worst = 0
    for sh in range(4):
        for off in range(32):
            worst = max(worst, _max_vector_byte_offset(off, 0, lmax, sh))
    assert worst < 2**32
    wraps = max(_max_vector_byte_offset(off, 0, lmax + 4, sh) for sh in range(4) for off in range(32))
    assert wraps >= 2**32
