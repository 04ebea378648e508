"""Shared helpers of the GPU tests: oracle-driven sessions replayed on the GPU.

Inputs always flow oracle -> GPU: drafts are chosen from the oracle's own
emitted tokens (or drawn by ``workloads``), never from GPU output, and the
GPU replays the same drafts step by step.
"""

import numpy as np

from oracle import OracleSession, match_reuse, top2_margin


def reuse_draft(generated, original, cursor, k):
    """Draft of the Reuse phase: the original tokens after the matched
    position, or after the cursor when nothing matches."""
    ds, _ = match_reuse(generated, original, cursor)
    start = ds if ds >= 0 else cursor
    return start, np.asarray(original[start:start + k], dtype=np.int32)


def oracle_reuse_session(shape, weights, prompt, original, steps, k):
    """Oracle-side Reuse session.  Returns the per-step drafts and results."""
    ref = OracleSession(shape, weights)
    ref.prefill(prompt)
    generated = [ref.pending]
    cursor = 0
    log = []
    for _ in range(steps):
        start, d = reuse_draft(generated, original, cursor, k)
        a, nxt, _ = ref.verify(d)
        log.append(dict(draft=d, a=a, next=nxt, logits=ref.last_logits.copy(), n=ref.n))
        generated += list(d[:a]) + [nxt]
        cursor = start + a + 1
    return ref, log


def deciding_margin(logits, a, k):
    """Smallest top-2 margin among the rows whose greedy token decided the
    outcome of an Eq. 7 acceptance: rows 0..min(a, k)."""
    m = top2_margin(logits)
    return float(m[:min(a, k) + 1].min())


def assert_step_matches(gpu_logits, gpu_a, gpu_next, ref_logits, ref_a, ref_next, k, tol):
    err = float(np.abs(gpu_logits - ref_logits).max())
    assert err <= tol, f"max |logit difference| {err} > {tol}"
    if deciding_margin(ref_logits, ref_a, k) > tol:
        assert (gpu_a, gpu_next) == (ref_a, ref_next)
        return True
    return (gpu_a, gpu_next) == (ref_a, ref_next)
