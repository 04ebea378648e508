"""Shared helpers of the GPU tests: oracle-driven sessions replayed on the GPU.

Inputs always flow oracle -> GPU: drafts are chosen from the oracle's own
emitted tokens (or drawn by ``workloads``), never from GPU output, and the
GPU replays the same drafts step by step.
"""

import numpy as np

from oracle import OracleSession, match_reuse, top2_margin
from oracle.numerics import round_bf16


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


def noise_probe(gen, rel):
    """Rounding-site hook of the oracle's forward: every value rounded to
    bf16 first carries a relative error rel * N(0, 1), the size of a float32
    evaluation's error.  The spread this causes in the logits is what the
    rounding sites leave open to any evaluation that is not the exact one."""
    def hook(site, layer, exact, rounded):
        return round_bf16(exact * (1.0 + rel * gen.standard_normal(np.shape(exact))))
    return hook


class OneLayer:
    """Weights of a one-layer model made of layer ``l`` of a full model (same
    embedding, LM head and final gain): a full-width test case that the
    oracle finishes in seconds."""

    def __init__(self, weights, l):
        self.embed, self.lm_head, self.final_gain = weights.embed, weights.lm_head, weights.final_gain
        self._w, self._l = weights, l
        self._layer = weights.layer(l)

    def layer(self, i):
        assert i == 0
        return self._layer


class RoundingCheck:
    """Oracle rounding-site hook that checks every bf16 value the GPU stored
    and follows it where it is a correct rounding.

    A bf16 pipeline rounds each value at the rounding sites; an evaluation in
    float32 carries a small error before it rounds, so where the exact value
    lies within that error of the midpoint between two bf16 numbers, either
    neighbour is a correct result (the "several results are correct" case).
    For each GPU value: equal to the oracle's rounding -> same; else, if it is
    the rounding of a value within ``delta`` of the exact one (delta = rel |x|
    + floor * rms of the row, rel = 2^-14 and floor = 2^-16 by default: a
    bound on a float32 evaluation's error, 2^-17 for the attention output's
    softmax weights, which enter the value product as a hi + lo pair of bf16
    numbers, about 2^-20 elsewhere, with room for cancellation) ->
    accepted near-tie flip; else -> mismatch (a kernel error).  The forward
    continues with the GPU's value where it is correct and with its own
    otherwise, so the logits that follow can be compared tightly: what is left
    is the float32 accumulation of the unrounded paths.

    gpu: {(site, layer): float64 array} of the GPU's stored values, one
    sequence's rows, shaped like the oracle's value at that site.
    """

    def __init__(self, gpu, rel=2.0 ** -14, floor=2.0 ** -16):
        self.gpu, self.rel, self.floor = gpu, rel, floor
        self.stats = {}       # (site, layer) -> [values, flips, mismatches]
        self.examples = []

    def __call__(self, site, layer, exact, rounded):
        g = self.gpu.get((site, layer))
        if g is None:
            return rounded
        g = np.asarray(g, dtype=np.float64).reshape(exact.shape)
        rows = exact.reshape(exact.shape[0], -1)
        rms = np.sqrt((rows * rows).mean(axis=1)).reshape((-1,) + (1,) * (exact.ndim - 1))
        delta = self.rel * np.abs(exact) + self.floor * rms
        same = g == rounded
        # rounding is monotone: the bf16 values between the roundings of
        # exact - delta and exact + delta are those of the values in between
        ok = same | ((g >= round_bf16(exact - delta)) & (g <= round_bf16(exact + delta)))
        st = self.stats.setdefault((site, layer), [0, 0, 0])
        st[0] += exact.size
        st[1] += int((ok & ~same).sum())
        st[2] += int((~ok).sum())
        if (~ok).any() and len(self.examples) < 5:
            i = np.argwhere(~ok)[0]
            self.examples.append((site, layer, tuple(int(x) for x in i), float(exact[tuple(i)]),
                                  float(g[tuple(i)]), float(rounded[tuple(i)])))
        return np.where(ok, g, rounded)

    def mismatches(self):
        return sum(v[2] for v in self.stats.values())

    def flips(self):
        return sum(v[1] for v in self.stats.values())

    def values(self):
        return sum(v[0] for v in self.stats.values())

    def summary(self):
        return (f"{self.values()} rounded values, {self.flips()} near-tie flips, "
                f"{self.mismatches()} mismatches {self.examples}")


def gpu_site_values(captured, shape, rows):
    """The captured rounding-site values of the block rows ``rows`` (a slice),
    as float64 arrays keyed like the oracle's rounding sites."""
    from oracle.numerics import to_f64
    return {key: to_f64(a[rows], shape.dtype) for key, a in captured.items()}


def valid_outcome(ref_logits, draft, a, nxt, err):
    """Whether a GPU outcome (a, next) is a correct greedy result for the
    oracle's logits when the GPU's logits are within err of them: every
    accepted draft token and the next token must be within 2 err of their
    row's maximum (a near tie that either evaluation may decide its way)."""
    lg = ref_logits
    for i in range(a):
        if lg[i][int(draft[i])] < lg[i].max() - 2 * err:
            return False
    return bool(lg[a][int(nxt)] >= lg[a].max() - 2 * err)


def adopt_outcome(ref, saved, draft, a, nxt):
    """Make the oracle session commit the GPU's outcome of a block it decided
    differently at a near tie: back to the state before the block, the
    pending row and draft[:a] committed, nxt pending."""
    ref.cache, ref.pending = saved
    ref.extend(np.asarray(draft[:a], dtype=np.int64))
    ref.pending = int(nxt)


def reuse_session_parity(eng, shape, weights, prompt, original, steps, k, tol, seq=0):
    """A Reuse session run side by side on the GPU (through the C ABI) and
    the oracle: each step's draft comes from the common generated stream and
    the matcher, both sides verify it, every logit is compared within tol and
    the outcome exactly.  Where the two decide a near tie differently (the
    deciding row's top-2 margin within the measured error), the GPU's outcome
    must be a correct one; the oracle then commits it and the session goes on
    (reading G12).  Returns (oracle session, steps compared, unpinned steps)."""
    ref = OracleSession(shape, weights)
    p_ref = ref.prefill(prompt)
    p_gpu = eng.prefill(seq, prompt)
    unpinned = 0
    lg = eng.logits()
    err = float(np.abs(lg - ref.last_logits[-len(lg):]).max())
    assert err <= tol, f"prefill: max |logit difference| {err} > {tol}"
    if p_gpu != p_ref:
        assert valid_outcome(ref.last_logits[-1:], [], 0, p_gpu, err)
        ref.pending = p_gpu
        unpinned += 1
    generated, cursor, compared = [ref.pending], 0, 0
    for _ in range(steps):
        start, d = reuse_draft(generated, original, cursor, k)
        saved = (ref.cache, ref.pending)
        ra, rn, _ = ref.verify(d)
        a, nxt, _ = eng.verify(seq, d)
        lg = eng.logits()
        err = float(np.abs(lg - ref.last_logits).max())
        assert err <= tol, f"max |logit difference| {err} > {tol}"
        if (a, nxt) != (ra, rn):
            assert deciding_margin(ref.last_logits, ra, len(d)) <= 2 * err, "a unique decision differs"
            assert valid_outcome(ref.last_logits, d, a, nxt, err), "the GPU's outcome is not a greedy one"
            adopt_outcome(ref, saved, d, a, nxt)
            unpinned += 1
        compared += 1
        assert eng.seq_state(seq) == (ref.n, ref.pending)
        generated += list(d[:a]) + [nxt]
        cursor = start + a + 1
    return ref, compared, unpinned
