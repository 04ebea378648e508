"""Oracle decoding session over its own KV cache (test infrastructure only).

Conventions (the paper leaves them open):
* The cache holds positions 0..n-1.  The last emitted token ("pending") has
  not been run through the model yet; it is row 0 of the next block, at
  position n.  ``prefill`` runs the prompt, commits all of it and emits the
  first pending token.
* ``verify`` runs [pending, d_1..d_K] (a chain, or a tree given parent
  pointers), accepts by Eq. 7 / the tree walk, commits the pending row plus
  the accepted rows in depth order (n -> n + 1 + a) and makes the emitted
  next token pending.  K = 0 is one plain greedy step of Eq. 1.
* ``extend`` commits [pending, tokens...] without verification (a draft
  model catching up with the accepted output).
* ``verify_topk`` is ``verify`` of a chain with the entropy-aware (or fixed)
  top-k acceptance of Eq. 9-10 in place of Eq. 7; ``score`` returns the
  logits of a chain block without committing anything.
* ``rollback`` truncates the committed cache to a shorter length and sets a
  new pending token.
"""

from __future__ import annotations

import numpy as np

from .accept import accept_linear, accept_tree, greedy_rows
from .entropy import accept_topk
from .model import chain_structure, forward_block, tree_structure


class OracleSession:
    def __init__(self, shape, weights, rounding=None):
        """rounding: None (the definition), or forward_block's rounding-site
        test hook, used by every forward of the session."""
        self.shape, self.weights = shape, weights
        self.rounding = rounding
        hk, hd = shape.n_kv_heads, shape.head_dim
        self.cache = [(np.zeros((0, hk, hd)), np.zeros((0, hk, hd))) for _ in range(shape.n_layers)]
        self.pending = None
        self.last_logits = None

    @property
    def n(self) -> int:
        return self.cache[0][0].shape[0]

    def _commit(self, block_kv, rows):
        rows = np.asarray(rows, dtype=np.int64)
        self.cache = [(np.concatenate([kc, k[rows]]), np.concatenate([vc, v[rows]]))
                      for (kc, vc), (k, v) in zip(self.cache, block_kv)]

    def set_cache(self, cache, pending):
        """Install an externally drawn committed cache (float64 values)."""
        self.cache = [(np.asarray(k, dtype=np.float64), np.asarray(v, dtype=np.float64)) for k, v in cache]
        self.pending = int(pending)

    def prefill(self, tokens):
        tokens = np.asarray(tokens, dtype=np.int64)
        depth, vis = chain_structure(len(tokens))
        logits, blk = forward_block(self.shape, self.weights, self.cache, tokens, depth, vis, self.rounding)
        self._commit(blk, np.arange(len(tokens)))
        self.pending = int(greedy_rows(logits[-1:])[0])
        self.last_logits = logits
        return self.pending

    def verify(self, draft, parent=None):
        """Returns (accept_len, next_token, accepted rows in depth order)."""
        if self.pending is None:
            raise RuntimeError("verify before prefill")
        draft = np.asarray(draft, dtype=np.int64)
        tokens = np.concatenate([[self.pending], draft])
        if parent is None:
            depth, vis = chain_structure(len(tokens))
        else:
            depth, vis = tree_structure(parent)
        logits, blk = forward_block(self.shape, self.weights, self.cache, tokens, depth, vis, self.rounding)
        g = greedy_rows(logits)
        if parent is None:
            a, nxt = accept_linear(draft, g)
            path = list(range(1, a + 1))
        else:
            a, nxt, path = accept_tree(draft, parent, g)
        self._commit(blk, [0] + path)
        self.pending = nxt
        self.last_logits = logits
        return a, nxt, path

    def extend(self, tokens):
        """Commit [pending, tokens...] without verification (a model following
        tokens chosen elsewhere); the greedy token after the last becomes
        pending and is returned."""
        rows = np.concatenate([[self.pending], np.asarray(tokens, dtype=np.int64)])
        depth, vis = chain_structure(len(rows))
        logits, blk = forward_block(self.shape, self.weights, self.cache, rows, depth, vis, self.rounding)
        self._commit(blk, np.arange(len(rows)))
        self.pending = int(greedy_rows(logits[-1:])[0])
        self.last_logits = logits
        return self.pending

    def score(self, draft):
        """Logits of the chain [pending, d_1..d_K]; the cache is unchanged."""
        tokens = np.concatenate([[self.pending], np.asarray(draft, dtype=np.int64)])
        depth, vis = chain_structure(len(tokens))
        logits, _ = forward_block(self.shape, self.weights, self.cache, tokens, depth, vis, self.rounding)
        return logits

    def verify_topk(self, draft, k: int, dynamic: bool = True):
        """Chain verification with the top-k acceptance of Eq. 9-10.
        Returns (accept_len, next_token, thresholds of the checked rows)."""
        if self.pending is None:
            raise RuntimeError("verify before prefill")
        draft = np.asarray(draft, dtype=np.int64)
        tokens = np.concatenate([[self.pending], draft])
        depth, vis = chain_structure(len(tokens))
        logits, blk = forward_block(self.shape, self.weights, self.cache, tokens, depth, vis, self.rounding)
        a, nxt, taus = accept_topk(draft, logits, k, dynamic)
        self._commit(blk, list(range(a + 1)))
        self.pending = nxt
        self.last_logits = logits
        return a, nxt, taus

    def greedy(self, steps: int):
        """Plain token-by-token greedy decoding (Eq. 1); returns emitted tokens."""
        out = []
        for _ in range(steps):
            _, nxt, _ = self.verify([])
            out.append(nxt)
        return out

    def rollback(self, new_len: int, pending: int):
        if not 0 <= new_len <= self.n:
            raise ValueError("rollback beyond the committed length")
        self.cache = [(k[:new_len], v[:new_len]) for k, v in self.cache]
        self.pending = int(pending)
