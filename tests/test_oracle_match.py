"""Pins of the oracle's Reuse matcher against brute force (CPU only)."""

import itertools

import numpy as np

from oracle import match_reuse


def _brute(gen, orig, cursor, lo, hi):
    """Enumerate every (L, j) pair; keep those that satisfy the matcher's
    conditions and pick the longest L, then the smallest j."""
    cands = []
    for ln in range(lo, hi + 1):
        if ln > len(gen):
            continue
        for j in range(len(orig)):
            if j + ln >= len(orig) or j + ln < cursor:
                continue
            if all(orig[j + i] == gen[len(gen) - ln + i] for i in range(ln)):
                cands.append((-ln, j))
    if not cands:
        return -1, 0
    ln, j = min(cands)
    return j - ln, -ln


def test_matcher_equals_brute_force_on_random_small_strings():
    g = np.random.default_rng(0)
    for _ in range(3000):
        orig = list(g.integers(0, 3, int(g.integers(0, 14))))
        gen = list(g.integers(0, 3, int(g.integers(0, 8))))
        cursor = int(g.integers(0, len(orig) + 2))
        lo = int(g.integers(1, 3))
        hi = int(g.integers(lo, 6))
        assert match_reuse(gen, orig, cursor, lo, hi) == _brute(gen, orig, cursor, lo, hi)


def test_matcher_resumes_right_after_the_consumed_prefix():
    orig = [5, 6, 7, 8, 9, 10, 11]
    # generated output ends with original[1:4] and the cursor is at 4
    assert match_reuse([1, 2, 6, 7, 8], orig, 4) == (4, 3)
    # after an insertion the last original token seen is re-found before the cursor
    assert match_reuse([5, 6, 99, 7], orig, 3) == (3, 1)
    # nothing in common
    assert match_reuse([42, 43], orig, 0) == (-1, 0)
    # a match whose draft would be empty is refused
    assert match_reuse([11], orig, 0) == (-1, 0)
    # the longest suffix wins over an earlier shorter one
    assert match_reuse([9, 7, 8], [7, 8, 1, 9, 7, 8, 2], 0) == (6, 3)
