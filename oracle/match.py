"""Prefix/suffix matcher that resumes Reuse (test infrastructure only).

Sec. "Reuse": when generation has to hand back to Reuse, positions in the
remaining original code whose preceding tokens match the suffix of what has
been generated become new draft starting points, and the original tokens from
there on are the next draft.

Reading used here (the paper fixes neither the n-gram length nor which
occurrence wins): try suffix lengths L from min(max_ngram, n_gen) down to
min_ngram; for the first L that matches anywhere, take the smallest j with
original[j : j+L] == generated[-L:], j + L >= cursor (the draft starts in the
remaining code) and j + L < len(original) (the draft is not empty).  Returns
(draft_start = j + L, L), or (-1, 0) when nothing matches.
"""


def match_reuse(generated, original, cursor: int, min_ngram: int = 1, max_ngram: int = 8):
    gen = [int(t) for t in generated]
    orig = [int(t) for t in original]
    n_gen, n_orig = len(gen), len(orig)
    for ln in range(min(max_ngram, n_gen), min_ngram - 1, -1):
        suffix = gen[n_gen - ln:]
        for j in range(max(0, cursor - ln), n_orig - ln):
            if orig[j:j + ln] == suffix:
                return j + ln, ln
    return -1, 0
