"""Entropy-aware dynamic and fixed top-k verification (ee_verify_topk,
Eq. 9-10) through the C ABI.

The oracle scores the same drafts in float64.  Drafts are built by the
oracle: each token is drawn at a random rank of the oracle's own row, so
that acceptance beyond the greedy token is exercised.  A decision is
compared where it is unique: the row's top k + 1 logits are separated by
more than twice the measured logit error, and k*H lies further from an
integer than the largest change that the error of the row's top-k logits
can cause (|d(kH)| <= 2k err to first order; 3k err is used).  The final norm gain is scaled so that rows
span low and high entropies.
"""

import numpy as np
import pytest

from helpers import adopt_outcome
from oracle import OracleSession, accept_topk, entropy_threshold, topk_tokens
from workloads import gen_weights, get_shape, planted_draft, zipf_tokens

pytestmark = pytest.mark.gpu

RANK_P = [0.45, 0.2, 0.12, 0.08, 0.06, 0.04, 0.03, 0.02]


@pytest.fixture(scope="module")
def ee():
    import paper_2506_02780_amd as mod
    return mod


def _model(cfg):
    if cfg == "f32":
        # 32000 columns: 16 chunks of 2048, the last one partial
        shape = get_shape("tiny", vocab=32000)
        w = gen_weights(shape, seed=21, std=0.1)
        w.final_gain = (w.final_gain * 4.0).astype(np.float32)
        return shape, w, 4 * 1e-4          # the stated fp32 tolerance, scaled with the logits
    shape = get_shape("tiny", n_layers=2, d_model=512, n_heads=4, n_kv_heads=2, head_dim=128, ffn=1024,
                      vocab=5024, dtype="bf16")   # 3 chunks, the last one partial
    w = gen_weights(shape, seed=22, std=0.02)
    w.final_gain = (w.final_gain * 8.0).astype(np.float32)   # a power of two: bf16 rounding unchanged
    return shape, w, 8 * 2e-2          # the stated bf16 tolerance, scaled with the logits


def _ranked_draft(ref, K, g):
    d = []
    for i in range(K):
        row = ref.score(d)[i]
        d.append(int(topk_tokens(row, 8)[g.choice(8, p=RANK_P)]))
    return np.asarray(d, dtype=np.int32)


def _row_unique(row, gpu_row, k, dynamic, err):
    s = np.sort(row)[::-1][:k + 1]
    if float(np.min(s[:-1] - s[1:])) <= 2 * err:
        return False
    if dynamic and k > 1:
        ids, h, _ = entropy_threshold(row, k)
        err_top = float(np.abs(gpu_row[ids] - row[ids]).max())
        x = k * h
        if abs(x - round(x)) <= 3 * k * err_top:
            return False
    return True


def _compare(gpu_res, gpu_logits, ref_logits, draft, k, dynamic, tol, seen):
    """Compare one step; returns False when a non-unique decision differed
    (the oracle then follows the GPU's outcome, reading G12)."""
    a, nxt, thr = gpu_res
    K = len(draft)
    err = float(np.abs(gpu_logits - ref_logits).max())
    assert err <= tol, f"max |logit difference| {err} > {tol}"
    print(f"K={K} err={err:.3g}", end="; ")
    unique = [_row_unique(ref_logits[i], gpu_logits[i], k, dynamic, err) for i in range(K + 1)]
    for i in range(K):
        tau = entropy_threshold(ref_logits[i], k, dynamic)[2]
        if unique[i]:
            assert thr[i] == tau, (i, thr[i], tau)
            seen.append(tau)
        assert 1 <= thr[i] <= k
    ra, rn, _ = accept_topk(draft, ref_logits, k, dynamic)
    if all(unique[:ra + 1]):
        assert (a, nxt) == (ra, rn)
        return True
    return (a, nxt) == (ra, rn)


@pytest.mark.parametrize("cfg,k,dynamic", [("f32", 3, True), ("f32", 5, True), ("f32", 5, False),
                                           ("f32", 8, True), ("bf16", 3, False), ("bf16", 5, True)])
def test_topk_session_matches_oracle(ee, cfg, k, dynamic):
    shape, w, tol = _model(cfg)
    prompt = zipf_tokens(shape.vocab, 80, seed=31)
    ref = OracleSession(shape, w)
    eng = ee.Engine(shape, w, max_ctx=256, k_max=12)
    assert eng.prefill(0, prompt) == ref.prefill(prompt)
    g = np.random.default_rng(k + 10 * dynamic)
    seen, compared, unpinned, accepted_beyond_greedy = [], 0, 0, 0
    # bf16 logits are ~0.04 apart from the oracle's, so few rows have a unique
    # dynamic threshold (k H must lie 3 k err from an integer): more steps
    steps = 8 if cfg == "f32" else 24
    for step in range(steps):
        K = int(g.integers(0, 13)) if step else 0
        draft = _ranked_draft(ref, K, g)
        res = eng.verify_topk([0], [draft], k, dynamic)[0]
        saved = (ref.cache, ref.pending)
        ra, rn, _ = ref.verify_topk(draft, k, dynamic)
        if not _compare(res, eng.logits(), ref.last_logits, draft, k, dynamic, tol, seen):
            # a near tie (rank or threshold) decided the GPU's way: the oracle
            # commits the GPU's outcome and the session goes on
            adopt_outcome(ref, saved, draft, res[0], res[1])
            unpinned += 1
            ra = res[0]
        compared += 1
        assert eng.seq_state(0) == (ref.n, ref.pending)
        accepted_beyond_greedy += sum(int(draft[i]) != int(np.argmax(ref.last_logits[i])) for i in range(ra))
    eng.close()
    print(f"{compared} steps compared, {unpinned} near ties followed, {len(seen)} thresholds compared, "
          f"values {sorted(set(seen))}")
    assert compared == steps
    if cfg == "f32":
        assert unpinned == 0
        assert len(seen) >= 30
        assert accepted_beyond_greedy >= 3
        if dynamic:
            assert len(set(seen)) >= 2
    else:
        assert unpinned <= steps // 3 and len(seen) >= 5


def _bf16_engine(ee, prompts, k_max=16):
    shape, w, _ = _model("bf16")
    eng = ee.Engine(shape, w, max_ctx=384, max_seqs=len(prompts), k_max=k_max)
    for b, p in enumerate(prompts):
        eng.prefill(b, p)
    return shape, w, eng


def _continuation(eng, seq, steps):
    """The sequence's own greedy continuation (K = 0 steps), rolled back."""
    n0, p0 = eng.seq_state(seq)
    out = [eng.verify(seq, [])[1] for _ in range(steps)]
    eng.rollback(seq, n0, p0)
    return out


def test_k1_is_greedy_verification_bitwise(ee):
    shape, w, eng = _bf16_engine(ee, [zipf_tokens(5024, 120, seed=41)])
    g = np.random.default_rng(2)
    for step in range(4):
        n0, p0 = eng.seq_state(0)
        truth = _continuation(eng, 0, 16)
        d = planted_draft(truth, int(g.integers(0, 16)), 15, shape.vocab, seed=step)
        a, n, _ = eng.verify(0, d)
        lg = eng.logits()
        kv = [eng.read_kv(0, l) for l in range(shape.n_layers)]
        for dyn in (True, False):
            eng.rollback(0, n0, p0)
            (a1, n1, thr), = eng.verify_topk([0], [d], 1, dyn)
            assert (a1, n1) == (a, n) and list(thr) == [1] * 15
            np.testing.assert_array_equal(eng.logits(), lg)
            for l in range(shape.n_layers):
                k1, v1 = eng.read_kv(0, l)
                np.testing.assert_array_equal(k1, kv[l][0])
                np.testing.assert_array_equal(v1, kv[l][1])
    eng.close()


def test_greedy_accepts_no_more_than_dynamic_and_dynamic_no_more_than_fixed(ee):
    shape, w, eng = _bf16_engine(ee, [zipf_tokens(5024, 150, seed=43)])
    ref = OracleSession(shape, w)
    ref.prefill(zipf_tokens(5024, 150, seed=43))
    g = np.random.default_rng(4)
    n0, p0 = eng.seq_state(0)
    strict = 0
    for step in range(6):
        d = _ranked_draft(ref, 12, g)
        a0, _, _ = eng.verify(0, d)
        lg = eng.logits()
        eng.rollback(0, n0, p0)
        (ad, _, thr_d), = eng.verify_topk([0], [d], 5, True)
        np.testing.assert_array_equal(eng.logits(), lg)
        eng.rollback(0, n0, p0)
        (af, _, thr_f), = eng.verify_topk([0], [d], 5, False)
        np.testing.assert_array_equal(eng.logits(), lg)
        eng.rollback(0, n0, p0)
        assert a0 <= ad <= af
        assert list(thr_f) == [5] * 12 and all(1 <= t <= 5 for t in thr_d)
        strict += (a0 < ad) + (ad < af)
    assert strict >= 1
    eng.close()


def test_batch_topk_equals_single_sequence_bitwise(ee):
    prompts = [zipf_tokens(5024, n, seed=50 + n) for n in (60, 130, 201)]
    shape, w, eng = _bf16_engine(ee, prompts)
    refs = []
    for p in prompts:
        r = OracleSession(shape, w)
        r.prefill(p)
        refs.append(r)
    g = np.random.default_rng(6)
    drafts = [_ranked_draft(r, 10, g) for r in refs]
    states = [eng.seq_state(b) for b in range(3)]
    single, logits, kvs = [], [], []
    for b in range(3):
        single.append(eng.verify_topk([b], [drafts[b]], 4, True)[0])
        logits.append(eng.logits())
        kvs.append([eng.read_kv(b, l) for l in range(shape.n_layers)])
        eng.rollback(b, *states[b])
    res = eng.verify_topk([2, 0, 1], [drafts[2], drafts[0], drafts[1]], 4, True)
    lg = eng.logits()
    for i, b in enumerate((2, 0, 1)):
        assert res[i][:2] == single[b][:2]
        np.testing.assert_array_equal(res[i][2], single[b][2])
        np.testing.assert_array_equal(lg[i * 11:(i + 1) * 11], logits[b])
        for l in range(shape.n_layers):
            k1, v1 = eng.read_kv(b, l)
            np.testing.assert_array_equal(k1, kvs[b][l][0])
            np.testing.assert_array_equal(v1, kvs[b][l][1])
    eng.close()


def test_topk_argument_errors_leave_state_unchanged(ee):
    shape, w, eng = _bf16_engine(ee, [zipf_tokens(5024, 50, seed=7)], k_max=8)
    before = eng.seq_state(0)
    for k in (0, 9, -1):
        with pytest.raises(ee.EEError) as e:
            eng.verify_topk([0], [[1, 2, 3]], k, True)
        assert e.value.code == ee.EE_EINVAL
    with pytest.raises(ee.EEError) as e:
        eng.verify_topk([0], [list(range(9))], 3, True)       # K > k_max
    assert e.value.code == ee.EE_EINVAL
    with pytest.raises(ee.EEError) as e:
        eng.verify_topk([0], [[1, 5024]], 3, True)            # token outside the vocabulary
    assert e.value.code == ee.EE_EINVAL
    assert eng.seq_state(0) == before
    (a, n, thr), = eng.verify_topk([0], [[]], 8, True)        # K = 0: one greedy step
    assert a == 0 and len(thr) == 0 and eng.seq_state(0) == (before[0] + 1, n)
    eng.close()
