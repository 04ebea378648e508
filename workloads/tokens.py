"""Seeded token streams, synthetic edits, draft trees and planted drafts.

Stand-ins for the paper's code-editing benchmarks, which are not available:
code-like token streams are Zipf(1.1) over the vocabulary (rank r has weight
r^-1.1, token id r-1); an "edit" replaces about 5% of the positions in spans
of 3 to 8 tokens, so roughly 95% of the edited output reuses the original,
inside the 50-100% reuse range the paper reports for its benchmarks.
"""

from __future__ import annotations

import math

import numpy as np


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def zipf_pmf(vocab: int, s: float = 1.1) -> np.ndarray:
    w = np.arange(1, vocab + 1, dtype=np.float64) ** (-s)
    return w / w.sum()


def zipf_tokens(vocab: int, n: int, seed: int = 42, s: float = 1.1) -> np.ndarray:
    """n token ids, rank-Zipf(s) over [0, vocab)."""
    g = _rng(seed)
    return g.choice(vocab, size=n, p=zipf_pmf(vocab, s)).astype(np.int32)


def inject_edits(tokens: np.ndarray, vocab: int, seed: int = 7, frac: float = 0.05,
                 span: tuple = (3, 8), s: float = 1.1):
    """Replace >= ceil(frac * N) positions in non-overlapping spans.

    Span lengths are uniform in [span[0], span[1]]; starts are uniform and
    redrawn when a span would touch an already-edited position.  Every
    replaced token is a fresh Zipf draw that differs from the original one.
    Returns (edited tokens, boolean mask of edited positions).
    """
    g = _rng(seed)
    tok = np.array(tokens, dtype=np.int32, copy=True)
    n = len(tok)
    need = math.ceil(frac * n)
    edited = np.zeros(n, dtype=bool)
    pmf = zipf_pmf(vocab, s)
    attempts = 0
    while edited.sum() < need:
        attempts += 1
        if attempts > 100000:
            raise RuntimeError("could not place edits")
        ln = int(g.integers(span[0], span[1] + 1))
        if ln > n:
            continue
        st = int(g.integers(0, n - ln + 1))
        lo, hi = max(0, st - 1), min(n, st + ln + 1)
        if edited[lo:hi].any():
            continue
        for p in range(st, st + ln):
            while True:
                t = int(g.choice(vocab, p=pmf))
                if t != tok[p]:
                    break
            tok[p] = t
        edited[st:st + ln] = True
    return tok, edited


def random_tree(k: int = 64, max_depth: int = 8, max_branch: int = 3, seed: int = 11,
                require_full_depth: bool = True) -> np.ndarray:
    """Parent pointers of a k-node draft tree (parent[i] < i, -1 = pending root).

    Node i picks its parent uniformly among the root and nodes 0..i-1 whose
    depth is below max_depth and which have fewer than max_branch children.
    The whole tree is redrawn until some node reaches max_depth.
    """
    g = _rng(seed)
    for _ in range(10000):
        parent = np.empty(k, dtype=np.int32)
        depth = np.empty(k, dtype=np.int32)
        nchild = np.zeros(k + 1, dtype=np.int32)      # index 0 = root, i+1 = node i
        for i in range(k):
            elig = [-1] if nchild[0] < max_branch else []
            elig += [j for j in range(i) if depth[j] < max_depth and nchild[j + 1] < max_branch]
            p = int(elig[int(g.integers(0, len(elig)))])
            parent[i] = p
            depth[i] = 1 if p < 0 else depth[p] + 1
            nchild[p + 1] += 1
        if not require_full_depth or k == 0 or depth.max() >= max_depth:
            return parent
    raise RuntimeError("no tree reached the requested depth")


def tree_tokens(parent: np.ndarray, chain_source, vocab: int, seed: int = 11,
                s: float = 1.1) -> np.ndarray:
    """Tokens for a draft tree.

    The first-child chain from the root (root's first child, its first child,
    ...) copies ``chain_source`` in order; every other node is a Zipf draw,
    redrawn until it differs from its siblings' tokens.
    """
    g = _rng(seed + 1)
    pmf = zipf_pmf(vocab, s)
    k = len(parent)
    tok = np.full(k, -1, dtype=np.int64)
    first_child = {}
    for i in range(k):
        first_child.setdefault(int(parent[i]), i)
    # walk the first-child chain
    cur, depth = -1, 0
    while cur in first_child and depth < len(chain_source):
        c = first_child[cur]
        tok[c] = int(chain_source[depth])
        cur, depth = c, depth + 1
    for i in range(k):
        if tok[i] >= 0:
            continue
        sib = {int(tok[j]) for j in range(k) if parent[j] == parent[i] and j != i and tok[j] >= 0}
        while True:
            t = int(g.choice(vocab, p=pmf))
            if t not in sib:
                break
        tok[i] = t
    # siblings that came from the chain source could collide with later draws only
    # through the loop above, which excludes them; chain-vs-chain collisions cannot occur.
    return tok.astype(np.int32)


def planted_draft(true_next, j: int, k: int, vocab: int, seed: int = 99,
                  s: float = 1.1) -> np.ndarray:
    """A k-token draft whose first j tokens are ``true_next[:j]`` and whose
    token j (when j < k) differs from ``true_next[j]``; the rest are Zipf."""
    assert 0 <= j <= k
    g = _rng(seed)
    pmf = zipf_pmf(vocab, s)
    d = g.choice(vocab, size=k, p=pmf).astype(np.int32)
    d[:j] = np.asarray(true_next[:j], dtype=np.int32)
    if j < k:
        while d[j] == true_next[j]:
            d[j] = int(g.choice(vocab, p=pmf))
    return d


def random_kv_context(n_layers: int, n: int, n_kv_heads: int, head_dim: int,
                      seed: int = 5, dtype: str = "bf16"):
    """Random committed K/V arrays, one [n, n_kv_heads, head_dim] pair per layer,
    N(0,1) values in the cache dtype (bf16 bit patterns or fp32)."""
    from .weights import _f32_to_bf16_bits
    g = _rng(seed)
    out = []
    for _ in range(n_layers):
        kv = []
        for _ in range(2):
            a = g.standard_normal((n, n_kv_heads, head_dim), dtype=np.float32)
            kv.append(_f32_to_bf16_bits(a) if dtype == "bf16" else a)
        out.append(tuple(kv))
    return out
