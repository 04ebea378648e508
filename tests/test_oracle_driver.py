"""Pins of the oracle's edit-session driver (Reuse / Generate phases), CPU."""

import numpy as np
import pytest

from oracle import OracleEditSession, OracleSession
from oracle.driver import GENERATE, REUSE
from workloads import gen_weights, get_shape, inject_edits, zipf_tokens


def _setup(draft_kind, seed=5, n_prompt=40, n_out=90):
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=seed, std=0.1)
    prompt = zipf_tokens(shape.vocab, n_prompt, seed=seed + 1)
    ref = OracleSession(shape, w)
    ref.prefill(prompt)
    greedy = [ref.pending] + ref.greedy(n_out - 1)
    original, _ = inject_edits(np.asarray(greedy, dtype=np.int32), shape.vocab, seed=7, frac=0.15)
    tgt = OracleSession(shape, w)
    tgt.prefill(prompt)
    draft = None
    if draft_kind == "same":
        draft = OracleSession(shape, w)
        draft.prefill(prompt)
    elif draft_kind == "other":
        dshape = get_shape("tiny", n_layers=1)
        draft = OracleSession(dshape, gen_weights(dshape, seed=seed + 100, std=0.1))
        draft.prefill(prompt)
    return tgt, draft, greedy, list(original), len(prompt)


def _run(sess, n):
    phases = []
    while len(sess.out) < n:
        ph, new = sess.step()
        phases.append((ph, len(new)))
    return phases


@pytest.mark.parametrize("draft_kind", [None, "same", "other"])
def test_greedy_verification_reproduces_greedy_decoding(draft_kind):
    """Eq. 7 in both phases: the output is the target's own greedy decoding
    (Eq. 1) whatever drafts the original code or the draft model propose."""
    tgt, draft, greedy, original, P = _setup(draft_kind)
    s = OracleEditSession(tgt, original, draft, k_reuse=8, gamma=4, top_k=0, min_match=3)
    phases = _run(s, len(greedy))
    assert s.out[:len(greedy)] == greedy
    assert {p for p, _ in phases} == {REUSE, GENERATE}       # edits send it to Generate and back
    if draft is not None:
        # the draft model follows the output: committed = prompt + out[:d_at], pending = out[d_at]
        assert draft.n == P + s.d_at and draft.pending == s.out[s.d_at]


def test_a_draft_model_equal_to_the_target_is_always_accepted():
    tgt, draft, greedy, original, _ = _setup("same")
    s = OracleEditSession(tgt, original, draft, k_reuse=8, gamma=4, top_k=0, min_match=3)
    gen_steps = [n for p, n in _run(s, len(greedy)) if p == GENERATE]
    assert gen_steps and all(n == 5 for n in gen_steps)       # gamma accepted + the target's token


def test_unedited_original_is_reused_in_full_blocks():
    tgt, _, greedy, _, _ = _setup(None)
    s = OracleEditSession(tgt, greedy, None, k_reuse=8, top_k=0)
    phases = _run(s, len(greedy) - 9)
    assert all(p == REUSE and n == 9 for p, n in phases)      # 8 reused + the bonus token each step


def test_top1_verification_is_greedy_verification():
    tgt, draft, greedy, original, _ = _setup("other", seed=9)
    s = OracleEditSession(tgt, original, draft, k_reuse=8, gamma=4, top_k=1, dynamic=True, min_match=3)
    _run(s, len(greedy))
    assert s.out[:len(greedy)] == greedy


def test_entropy_aware_generate_accepts_at_least_as_much_as_greedy():
    """Same draft proposals, relaxed acceptance: the first Generate step with a
    5-token top-k accepts at least as many draft tokens as greedy."""
    res = {}
    for k in (0, 5):
        tgt, draft, greedy, original, _ = _setup("other", seed=11)
        s = OracleEditSession(tgt, original, draft, k_reuse=8, gamma=4, top_k=k, dynamic=False, min_match=3)
        while True:
            ph, new = s.step()
            if ph == GENERATE:
                res[k] = len(new)
                break
    assert res[5] >= res[0]
