"""Greedy decoding and acceptance (test infrastructure only).

Sec. "Reuse", Eq. 7: with decode = greedy (argmax), draft token d_i is
accepted while decode(p_i) = d_i for all i <= j; the accepted length is the
largest such j.  p_i, the distribution that decides d_i, is produced by the
row that precedes d_i in the block [pending, d_1 .. d_K] (row 0 is the
pending token).  After the accepted prefix the target's own greedy token at
the last accepted row is emitted: a correction when a draft token was
rejected, the bonus token of the all-accepted case (Sec. "Speculative
Decoding": M+1 tokens from one forward).

A draft tree (rows 1..K are nodes with parent pointers) is accepted by the
greedy walk: from the pending row, step to the lowest-indexed child whose
token equals the current row's greedy token, until no child does.
"""

import numpy as np


def greedy_rows(logits):
    """Greedy token of every row; the lowest index wins an exact tie."""
    return np.argmax(np.asarray(logits), axis=1).astype(np.int64)


def top2_margin(logits):
    """Largest minus second-largest logit of every row."""
    s = np.sort(np.asarray(logits, dtype=np.float64), axis=1)
    return s[:, -1] - s[:, -2]


def accept_linear(draft, g):
    """draft: [K] tokens d_1..d_K; g: [K+1] greedy tokens of rows 0..K.
    Returns (accepted length a, next token g[a])."""
    a = 0
    while a < len(draft) and int(draft[a]) == int(g[a]):
        a += 1
    return a, int(g[a])


def accept_tree(node_tokens, parent, g):
    """node_tokens[i], parent[i] for nodes i (row i+1; parent -1 = row 0).
    Returns (a, next token, accepted rows in depth order)."""
    k = len(node_tokens)
    cur, path = 0, []
    while True:
        nxt = None
        for i in range(k):
            if int(parent[i]) + 1 == cur and int(node_tokens[i]) == int(g[cur]):
                nxt = i + 1
                break
        if nxt is None:
            break
        path.append(nxt)
        cur = nxt
    return len(path), int(g[cur]), path
