"""Pins of the oracle's entropy-aware and fixed top-k verification (CPU)."""

import math

import numpy as np
import pytest
from scipy.stats import entropy as scipy_entropy

from oracle import accept_linear, accept_topk, entropy_threshold, greedy_rows, topk_tokens


def test_topk_ranks_by_score_then_lower_id():
    row = np.array([0.5, 2.0, 2.0, -1.0, 2.0, 1.0])
    assert list(topk_tokens(row, 4)) == [1, 2, 4, 5]
    g = np.random.default_rng(0)
    for _ in range(50):
        r = np.round(g.normal(size=40), 1)          # many exact ties
        k = int(g.integers(1, 9))
        brute = sorted(range(40), key=lambda i: (-r[i], i))[:k]
        assert list(topk_tokens(r, k)) == brute


@pytest.mark.parametrize("k", [2, 3, 5, 8])
def test_uniform_top_k_gives_full_threshold_and_one_hot_gives_one(k):
    row = np.full(100, -5.0)
    row[[3, 17, 40, 41, 42, 60, 70, 90][:k]] = 2.0
    _, h, tau = entropy_threshold(row, k)
    assert h == pytest.approx(1.0, abs=1e-12) and tau == k
    row = np.zeros(100)
    row[7] = 60.0                                     # the others carry ~e^-60
    _, h, tau = entropy_threshold(row, k)
    assert h < 1e-20 and tau == 1


def test_two_point_closed_form():
    for p in (0.5, 0.6, 0.75, 0.9, 0.99):
        row = np.array([math.log(p), math.log(1 - p), -30.0, -30.0])
        _, h, tau = entropy_threshold(row, 2)
        hb = -(p * math.log(p) + (1 - p) * math.log(1 - p)) / math.log(2)
        assert h == pytest.approx(hb, rel=1e-9)
        assert tau == max(1, math.ceil(2 * hb))


def test_entropy_matches_an_independent_routine_and_is_shift_invariant():
    g = np.random.default_rng(1)
    for _ in range(200):
        k = int(g.integers(2, 9))
        row = g.normal(scale=float(g.choice([0.1, 1.0, 4.0])), size=64)
        ids, h, tau = entropy_threshold(row, k)
        p = np.exp(row - row.max())
        p = p / p.sum()
        q = p[ids] / p[ids].sum()                     # renormalised top-k probabilities
        assert h == pytest.approx(scipy_entropy(q, base=k), abs=1e-12)
        assert 0.0 <= h <= 1.0 + 1e-12
        assert tau == min(k, max(1, math.ceil(k * h)))
        _, h2, tau2 = entropy_threshold(row + 3.25, k)
        assert h2 == pytest.approx(h, abs=1e-12) and tau2 == tau


def test_flatter_rows_get_larger_thresholds():
    g = np.random.default_rng(2)
    row = g.normal(size=64)
    taus = [entropy_threshold(row / temp, 5)[2] for temp in (0.05, 0.2, 1.0, 5.0, 50.0)]
    assert taus == sorted(taus) and taus[0] == 1 and taus[-1] == 5


def test_fixed_mode_uses_k():
    g = np.random.default_rng(3)
    for k in (2, 3, 5):
        assert entropy_threshold(g.normal(size=50), k, dynamic=False)[2] == k


def test_k1_is_greedy_verification_and_larger_k_accepts_at_least_as_much():
    g = np.random.default_rng(4)
    for _ in range(100):
        K, V = int(g.integers(0, 9)), 30
        logits = g.normal(size=(K + 1, V))
        gr = greedy_rows(logits)
        # drafts that follow the greedy tokens for a while, then the 2nd-5th best
        draft = [int(gr[i]) if g.random() < 0.6 else int(topk_tokens(logits[i], 5)[int(g.integers(1, 5))])
                 for i in range(K)]
        a1, n1, _ = accept_topk(draft, logits, 1)
        assert (a1, n1) == accept_linear(draft, gr)
        for dyn in (True, False):
            a, n, taus = accept_topk(draft, logits, 5, dyn)
            assert a >= a1 and n == int(gr[a])
            # brute force: a is the first row whose draft token ranks beyond its threshold
            ranks = [list(topk_tokens(logits[i], V)).index(draft[i]) for i in range(K)]
            ths = [entropy_threshold(logits[i], 5, dyn)[2] for i in range(K)]
            first = next((i for i in range(K) if ranks[i] >= ths[i]), K)
            assert a == first and taus == ths[:min(K, a + 1)]


def test_token_at_rank_tau_is_accepted_and_at_tau_plus_one_rejected():
    g = np.random.default_rng(5)
    hits = 0
    for _ in range(300):
        row = g.normal(scale=float(g.choice([0.5, 2.0, 5.0])), size=40)
        ids, _, tau = entropy_threshold(row, 5)
        logits = np.stack([row, g.normal(size=40)])
        assert accept_topk([int(ids[tau - 1])], logits, 5)[0] == 1
        if tau < 5:
            assert accept_topk([int(ids[tau])], logits, 5)[0] == 0
            hits += 1
    assert hits > 20
