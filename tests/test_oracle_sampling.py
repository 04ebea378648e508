"""Pins of the oracle's stochastic speculative sampling (Eq. 4), CPU."""

import numpy as np
import pytest

from oracle import accept_sample, sample_index, target_probs

GRID = 4000
MID = (np.arange(GRID) + 0.5) / GRID      # midpoints of a uniform grid on [0, 1)


def _first_token_distribution(p_logits, q, residual):
    """Distribution of the first emitted token of a K = 1 block when d ~ q,
    eps ~ U[0,1) and u ~ U[0,1), from calls of accept_sample on grids."""
    V = len(q)
    logits = np.stack([p_logits, np.zeros(V)])
    out = np.zeros(V)
    for d in range(V):
        if q[d] == 0:
            continue
        acc = np.mean([accept_sample([d], logits, [e, 0.0], [0.5, 0.5], [q])[0] == 1 for e in MID[::10]])
        res = np.zeros(V)
        if acc < 1:                               # a rejection is possible: eps just below 1 forces it
            for u in MID:
                a, t = accept_sample([d], logits, [1 - 1e-12, 0.0], [u, 0.5], [q], residual=residual)
                assert a == 0
                res[t] += 1.0 / GRID
        out += q[d] * (acc * np.eye(V)[d] + (1 - acc) * res)
    return out


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_residual_resampling_reproduces_the_target_distribution(seed):
    g = np.random.default_rng(seed)
    V = 5
    pl = g.normal(scale=1.5, size=V)
    q = g.dirichlet(np.ones(V))
    p = target_probs(pl)
    np.testing.assert_allclose(_first_token_distribution(pl, q, True), p, atol=3e-3)


def test_resampling_from_p_gives_the_mixture_the_paper_describes():
    g = np.random.default_rng(5)
    V = 4
    pl = g.normal(size=V)
    q = g.dirichlet(np.ones(V))
    p = target_probs(pl)
    m = np.minimum(p, q)
    expect = m + (1 - m.sum()) * p            # keep d with prob min(1, p/q), else draw from p
    np.testing.assert_allclose(_first_token_distribution(pl, q, False), expect, atol=3e-3)


def test_sample_index_is_the_inverse_cdf():
    g = np.random.default_rng(3)
    for _ in range(200):
        w = g.random(7) * (g.random(7) > 0.3)
        if w.sum() == 0:
            continue
        u = g.random()
        acc, v = 0.0, 0
        while acc + w[v] <= u * w.sum():
            acc += w[v]
            v += 1
        assert sample_index(w, u) == v


def test_equal_distributions_accept_everything_and_the_bonus_is_drawn_from_the_last_row():
    g = np.random.default_rng(4)
    logits = g.normal(size=(4, 6))
    q = [target_probs(logits[i]) for i in range(3)]
    for e in (0.0, 0.5, 0.999):
        a, t = accept_sample([1, 2, 3], logits, [e] * 3, [0.1, 0.2, 0.3, 0.7], q)
        assert a == 3 and t == sample_index(target_probs(logits[3]), 0.7)


def test_greedy_draft_at_low_temperature_is_greedy_verification():
    g = np.random.default_rng(6)
    logits = g.normal(size=(5, 20)) * 3
    greedy = logits.argmax(axis=1)
    draft = [int(greedy[0]), int(greedy[1]), (int(greedy[2]) + 1) % 20, 0]
    a, t = accept_sample(draft, logits, [0.9] * 4, [0.3] * 5, None, temperature=1e-3)
    assert a == 2 and t == greedy[2]


def test_temperature_flattens_and_sharpens():
    row = np.array([2.0, 1.0, 0.0])
    assert target_probs(row, 1e6)[0] == pytest.approx(1 / 3, abs=1e-5)
    np.testing.assert_allclose(target_probs(row, 0.5), np.exp(2 * row) / np.exp(2 * row).sum())
