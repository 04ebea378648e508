"""Oracle edit-session driver: the Reuse / Generate phase machine.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. "Reuse": the original code c serves as the draft; the target verifies it
greedily (Eq. 7); a rejection marks an edit position and hands over to the
Generate phase; prefix matching between the remaining c and the generated
suffix resumes Reuse.  Sec. "Generate": a draft model proposes gamma tokens
and the target verifies them greedily or with the entropy-aware rule of
Eq. 9-10.  Readings used (the paper leaves them open):
* the Reuse draft starts after the match of the output's suffix in c (at or
  after the cursor; while the output is shorter than the shortest suffix
  length, the whole output is matched), else at the cursor; after a step the cursor moves past
  the accepted tokens and the rejected one (substitution);
* a Reuse step with a rejection switches to Generate, a fully accepted one
  stays in Reuse; a Reuse step with nothing left in c runs as Generate;
* after a Generate step the matcher runs; a match switches to Reuse;
* the draft model follows the output: before drafting it commits the output
  tokens it has not seen, drafting continues greedily from there, and it
  keeps only the accepted part afterwards.  Without a draft model a Generate
  step is one plain greedy step of the target.
"""

from __future__ import annotations

import numpy as np

from .accept import greedy_rows
from .match import match_reuse
from .session import OracleSession

REUSE, GENERATE = 0, 1


class OracleEditSession:
    def __init__(self, target: OracleSession, original, draft: OracleSession | None = None,
                 k_reuse=32, gamma=7, top_k=0, dynamic=True, min_match=3, max_match=8):
        self.t, self.d = target, draft
        self.c = [int(x) for x in original]
        self.k_reuse, self.gamma, self.top_k, self.dynamic = k_reuse, gamma, top_k, dynamic
        self.min_match, self.max_match = min_match, max_match
        self.out = [target.pending]
        self.phase, self.cursor = REUSE, 0
        if draft is not None:
            assert draft.n == target.n
            draft.pending = target.pending
        # output index of the draft model's pending token
        self.d_at = 0

    def _match(self):
        lo = min(self.min_match, len(self.out))
        return match_reuse(self.out, self.c, self.cursor, lo, max(lo, self.max_match))[0]

    def _verify(self, draft_tokens, entropy):
        if entropy and self.top_k:
            a, nxt, _ = self.t.verify_topk(draft_tokens, self.top_k, self.dynamic)
        else:
            a, nxt, _ = self.t.verify(draft_tokens)
        return a, nxt

    def step(self):
        phase = self.phase
        if phase == REUSE:
            ds = self._match()
            start = ds if ds >= 0 else min(self.cursor, len(self.c))
            d = self.c[start:start + self.k_reuse]
            if not d:
                phase = GENERATE
            else:
                a, nxt = self._verify(d, entropy=False)
                self.cursor = start + a + 1
                self.phase = GENERATE if a < len(d) else REUSE
        if phase == GENERATE:
            if self.d is None:
                d = []
                a, nxt = self._verify([], entropy=False)
            else:
                m = len(self.out) - 1
                # catch up: commit the output from the draft's pending token to out[m]
                first = self.d.extend(self.out[self.d_at + 1:m + 1])
                d = [first]
                for _ in range(self.gamma - 1):
                    _, g, _ = self.d.verify([])
                    d.append(g)
                n_before = self.t.n
                a, nxt = self._verify(d, entropy=True)
                if a < self.gamma:
                    # keep out[..m] and d_1..d_a; the target's token is pending
                    self.d.rollback(n_before + 1 + a, nxt)
                    self.d_at = m + a + 1
                else:
                    self.d_at = m + self.gamma          # d_gamma is the draft's pending token
            self.phase = GENERATE
        new = list(d[:a]) + [nxt]
        self.out += new
        if phase == GENERATE:
            if self._match() >= 0:
                self.phase = REUSE
        return phase, new
