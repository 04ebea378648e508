"""Entropy-aware dynamic verification and fixed top-k verification
(test infrastructure only).

Sec. "Edit" (Eq. 9 and 10): at the row that precedes a draft token, take
the target's k largest probabilities (the base threshold k; ties ranked by
the lower token index) and their normalised entropy

    H_norm = -sum_i q_i log q_i / log k,   i = 1..k,

where q are those k probabilities renormalised to sum to one (reading: the
entropy is that of the top-k distribution, so H_norm lies in [0, 1]; since
q_i = exp(l_i - l_1) / sum_j exp(l_j - l_1) only the top-k logits are
needed).  The acceptance threshold is top_tau = ceil(k H_norm), or 1 when
that is below 1 (Eq. 10), and the draft token is accepted when it is among
the target's top_tau tokens.  The fixed top-k verification of the paper's
comparison accepts when the draft token is among the top k.  With k = 1
both are greedy verification.  Unlike greedy verification these rules are
not lossless: an accepted token need not be the target's argmax.

After the accepted prefix the target's own greedy token of the last
accepted row is emitted, as in greedy verification.
"""

import math

import numpy as np


def topk_tokens(row, k: int) -> np.ndarray:
    """The k highest-scoring token ids of one row, best first; equal scores
    are ranked by the lower token id."""
    row = np.asarray(row, dtype=np.float64)
    order = np.lexsort((np.arange(len(row)), -row))   # primary: -score, then id
    return order[:k]


def entropy_threshold(row, k: int, dynamic: bool = True):
    """(top-k token ids, H_norm, top_tau) of one row of logits."""
    ids = topk_tokens(row, k)
    if k == 1:
        return ids, 0.0, 1
    v = np.asarray(row, dtype=np.float64)[ids]
    q = np.exp(v - v[0])
    q = q / q.sum()
    nz = q[q > 0]
    h = float(-(nz * np.log(nz)).sum() / math.log(k))
    if not dynamic:
        return ids, h, k
    tau = max(1, math.ceil(k * h))
    return ids, h, min(tau, k)


def accept_topk(draft, logits, k: int, dynamic: bool = True):
    """draft: [K] tokens; logits: [K+1, V] rows 0..K of the verify block.
    Returns (accepted length a, next token = greedy token of row a, the
    top_tau of every row that was checked)."""
    logits = np.asarray(logits)
    a, taus = 0, []
    while a < len(draft):
        ids, _, tau = entropy_threshold(logits[a], k, dynamic)
        taus.append(tau)
        if int(draft[a]) not in set(int(x) for x in ids[:tau]):
            break
        a += 1
    return a, int(np.argmax(logits[a])), taus
