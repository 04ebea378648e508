"""Stochastic speculative sampling (Sec. "Speculative Decoding", Eq. 4).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The target's distribution of row i is p_i = softmax(logits_i / temperature).
Draft token d_{i+1} (proposed from the draft distribution q_i) is accepted when
the uniform draw eps_i is below p_i[d] / q_i[d] (taken as eps_i q_i[d] <
p_i[d], which needs no division); the first rejection ends the block.  At the
rejected row a token is resampled; when every draft token is accepted, the bonus token is sampled from the last row's p.  Readings (the
paper is terse here):
* resampling after a rejection uses the residual max(0, p_a - q_a),
  renormalised (`residual=True`: the standard rule, which makes the output
  distribution exactly p), or p_a itself as the paper's sentence reads
  (`residual=False`);
* q = None means a greedy draft model: q_i is one-hot at d_{i+1};
* sampling draws token v with the smallest index whose cumulative weight (in
  token order) exceeds u * total, u uniform in [0, 1); the random numbers are
  inputs (eps[K], u[K + 1]), so every draw is reproducible.
All arithmetic is float64.
"""

from __future__ import annotations

import numpy as np


def target_probs(logits_row, temperature=1.0):
    x = np.asarray(logits_row, dtype=np.float64) / float(temperature)
    e = np.exp(x - x.max())
    return e / e.sum()


def sample_index(weights, u):
    """Smallest v with cumsum(weights)[v] > u * sum(weights)."""
    w = np.asarray(weights, dtype=np.float64)
    c = np.cumsum(w)
    return int(np.searchsorted(c, u * c[-1], side="right"))


def accept_sample(draft, logits, eps, u, q=None, temperature=1.0, residual=True):
    """Returns (accept_len, next_token)."""
    draft = [int(t) for t in draft]
    K = len(draft)
    for i in range(K):
        p = target_probs(logits[i], temperature)
        d = draft[i]
        qd = 1.0 if q is None else float(q[i][d])
        if eps[i] * qd < p[d]:
            continue
        if residual:
            qi = np.zeros_like(p) if q is None else np.asarray(q[i], dtype=np.float64)
            if q is None:
                qi[d] = 1.0
            w = np.maximum(p - qi, 0.0)
            if w.sum() <= 0:          # p == q: nothing left to correct; fall back to p
                w = p
        else:
            w = p
        return i, sample_index(w, u[i])
    return K, sample_index(target_probs(logits[K], temperature), u[K])
