"""Long linear drafts (K up to 512 rows in one block) through the C ABI.

A Reuse draft needs no fixed length (Sec. "Reuse": one forward can verify a
long span of the original code), so a block may hold up to 513 rows.  The
oracle checks planted drafts exactly; the GPU's own properties (rows equal
to those of short blocks bit for bit, the speculative stream equal to the
greedy stream) are checked at the bf16 shape.
"""

import numpy as np
import pytest

from oracle import OracleSession, entropy_threshold
from tests.helpers import assert_step_matches
from workloads import gen_weights, get_shape, planted_draft, zipf_tokens

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ee():
    import paper_2506_02780_amd as mod
    return mod


def _bf16_small(**kw):
    base = dict(n_layers=2, d_model=512, n_heads=4, n_kv_heads=2, head_dim=128, ffn=1024,
                vocab=2048, dtype="bf16")
    base.update(kw)
    return get_shape("tiny", **base)


def test_long_planted_drafts_accept_exactly(ee):
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=91, std=0.1)
    prompt = zipf_tokens(shape.vocab, 50, seed=3)
    ref = OracleSession(shape, w)
    ref.prefill(prompt)
    eng = ee.Engine(shape, w, max_ctx=2048, k_max=512)
    eng.prefill(0, prompt)
    g = np.random.default_rng(1)
    for K in (100, 512, 257, 300):
        probe = OracleSession(shape, w)
        probe.set_cache(ref.cache, ref.pending)
        truth = probe.greedy(K + 1)
        j = int(g.integers(K // 2, K + 1))
        d = planted_draft(truth, j, K, shape.vocab, seed=K)
        ra, rn, _ = ref.verify(d)
        a, n, _ = eng.verify(0, d)
        assert_step_matches(eng.logits(), a, n, ref.last_logits, ra, rn, K, 1e-4)
        assert ra == j and eng.seq_state(0) == (ref.n, ref.pending)
    for l in range(shape.n_layers):
        k, v = eng.read_kv(0, l)
        np.testing.assert_allclose(k, ref.cache[l][0], rtol=0, atol=2e-5)
        np.testing.assert_allclose(v, ref.cache[l][1], rtol=0, atol=2e-5)
    eng.close()


@pytest.mark.parametrize("width", [512, 4096, 7168])
def test_long_block_rows_equal_short_block_rows_bitwise(ee, width):
    """Rows of a 401-row block equal the same rows computed one block at a
    time (K = 0 steps) bit for bit: logits and the committed K/V.  The block's
    down projection and LM head (and at width 7168 every projection) run in
    six 80-row groups, the single rows in a launch of one row.  Width 4096
    (one layer): two K slices in the LM head, and the gate/up kernel a single
    pass over d, in 32-row groups at 401 rows and one row alone.  Width 7168
    (one layer): four K slices of 56 super-steps (7 per wave, the eighth slot
    of each wave zero) in the QKV, O, gate/up projections and the LM head,
    and a 7-super-step down projection (FFN 224: one wave without
    super-steps)."""
    if width == 512:
        shape = _bf16_small()
    elif width == 4096:
        shape = _bf16_small(n_layers=1, d_model=4096, n_heads=32, n_kv_heads=8, ffn=2048)
    else:
        shape = _bf16_small(n_layers=1, d_model=7168, n_heads=56, n_kv_heads=8, ffn=224)
    w = gen_weights(shape, seed=92, std=0.05 if width == 512 else 0.02)
    prompt = zipf_tokens(shape.vocab, 130, seed=4)
    eng = ee.Engine(shape, w, max_ctx=1024, k_max=512)
    eng.prefill(0, prompt)
    n0, p0 = eng.seq_state(0)
    steps = []
    for _ in range(401):
        steps.append((eng.verify(0, [])[1], eng.logits()[0].copy()))
    kv_ref = [eng.read_kv(0, l) for l in range(shape.n_layers)]
    eng.rollback(0, n0, p0)
    draft = [t for t, _ in steps[:400]]
    a, nxt, _ = eng.verify(0, draft)
    assert a == 400 and nxt == steps[400][0]
    lg = eng.logits()
    for i in range(401):
        np.testing.assert_array_equal(lg[i], steps[i][1])
    for l in range(shape.n_layers):
        k, v = eng.read_kv(0, l)
        np.testing.assert_array_equal(k, kv_ref[l][0])
        np.testing.assert_array_equal(v, kv_ref[l][1])
    eng.close()


def test_long_drafts_stream_equals_greedy_stream(ee):
    shape = _bf16_small()
    w = gen_weights(shape, seed=93, std=0.05)
    prompt = zipf_tokens(shape.vocab, 90, seed=5)
    eng = ee.Engine(shape, w, max_ctx=2048, k_max=512)
    eng.prefill(0, prompt)
    n0, p0 = eng.seq_state(0)
    target = [eng.verify(0, [])[1] for _ in range(1100)]
    eng.rollback(0, n0, p0)
    out = []
    g = np.random.default_rng(7)
    while len(out) < 1000:
        rest = target[len(out):]
        K = int(g.choice([128, 256, 512]))
        j = min(int(g.integers(0, K + 1)), len(rest))
        d = planted_draft(rest, j, K, shape.vocab, seed=int(g.integers(1 << 30)))
        a, nxt, _ = eng.verify(0, d)
        assert a == j
        out += list(d[:a]) + [nxt]
    assert out[:1000] == target[:1000]
    eng.close()


def test_long_topk_thresholds_match_oracle(ee):
    """Entropy-aware verification over a 201-row block: every unique
    threshold equals the oracle's (sharpened fp32 model)."""
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=94, std=0.1)
    w.final_gain = (w.final_gain * 4.0).astype(np.float32)
    prompt = zipf_tokens(shape.vocab, 60, seed=6)
    ref = OracleSession(shape, w)
    ref.prefill(prompt)
    eng = ee.Engine(shape, w, max_ctx=512, k_max=256)
    eng.prefill(0, prompt)
    d = zipf_tokens(shape.vocab, 200, seed=8)
    (a, nxt, thr), = eng.verify_topk([0], [d], 5, True)
    ref_logits = ref.score(d)
    gl = eng.logits()
    err = float(np.abs(gl - ref_logits).max())
    assert err <= 1e-3
    compared = 0
    for i in range(200):
        ids, h, tau = entropy_threshold(ref_logits[i], 5)
        s = np.sort(ref_logits[i])[::-1][:6]
        x = 5 * h
        if np.min(s[:-1] - s[1:]) > 2 * err and abs(x - round(x)) > 15 * err:
            assert thr[i] == tau, (i, thr[i], tau)
            compared += 1
    assert compared >= 150
    eng.close()


def test_trees_stay_within_64_nodes(ee):
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=3)
    eng = ee.Engine(shape, w, max_ctx=512, k_max=128)
    eng.prefill(0, zipf_tokens(shape.vocab, 20, seed=1))
    before = eng.seq_state(0)
    with pytest.raises(ee.EEError) as e:
        eng.verify(0, list(range(65)), list(range(-1, 64)))
    assert e.value.code == ee.EE_EINVAL
    assert eng.seq_state(0) == before
    a, _, nodes = eng.verify(0, list(range(64)), list(range(-1, 63)))   # a 64-node chain is fine
    assert eng.seq_state(0)[0] == before[0] + 1 + a
    eng.close()


def test_long_batch_rows_equal_single_sequence_rows_bitwise(ee):
    """Two sequences with 200-token drafts in one block (wide attention and
    row-group GEMMs) equal each sequence verified alone, bit for bit."""
    shape = _bf16_small()
    w = gen_weights(shape, seed=95, std=0.05)
    prompts = [zipf_tokens(shape.vocab, n, seed=9 + n) for n in (90, 333)]
    eng = ee.Engine(shape, w, max_ctx=1024, max_seqs=2, k_max=256)
    for b, p in enumerate(prompts):
        eng.prefill(b, p)
    states = [eng.seq_state(b) for b in range(2)]
    drafts = [zipf_tokens(shape.vocab, 200, seed=20 + b) for b in range(2)]
    single = []
    for b in range(2):
        res = eng.verify(b, drafts[b])
        single.append((res[:2], eng.logits(), [eng.read_kv(b, l) for l in range(shape.n_layers)]))
        eng.rollback(b, *states[b])
    res = eng.verify_batch([1, 0], [drafts[1], drafts[0]])
    lg = eng.logits()
    for i, b in enumerate((1, 0)):
        assert res[i][:2] == single[b][0]
        np.testing.assert_array_equal(lg[i * 201:(i + 1) * 201], single[b][1])
        for l in range(shape.n_layers):
            k, v = eng.read_kv(b, l)
            np.testing.assert_array_equal(k, single[b][2][l][0])
            np.testing.assert_array_equal(v, single[b][2][l][1])
    eng.close()


def test_extend_commits_every_row_and_matches_oracle(ee):
    """ee_extend: [pending, tokens...] committed without verification, in
    blocks of k_max + 1 rows; the new pending token and the cache match the
    oracle, and n = 0 is a plain greedy step."""
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=96, std=0.1)
    prompt = zipf_tokens(shape.vocab, 30, seed=2)
    ref = OracleSession(shape, w)
    ref.prefill(prompt)
    eng = ee.Engine(shape, w, max_ctx=512, k_max=16)
    eng.prefill(0, prompt)
    for n in (0, 5, 16, 17, 40):          # 40 rows + pending: three blocks of <= 17 rows
        toks = zipf_tokens(shape.vocab, n, seed=n + 3)
        assert eng.extend(0, toks) == ref.extend(toks)
        assert eng.seq_state(0) == (ref.n, ref.pending)
    for l in range(shape.n_layers):
        k, v = eng.read_kv(0, l)
        np.testing.assert_allclose(k, ref.cache[l][0], rtol=0, atol=2e-5)
        np.testing.assert_allclose(v, ref.cache[l][1], rtol=0, atol=2e-5)
    n0, p0 = eng.seq_state(0)
    a, nxt, _ = eng.verify(0, [])
    eng.rollback(0, n0, p0)
    assert eng.extend(0, []) == nxt
    with pytest.raises(ee.EEError) as e:
        eng.extend(0, [shape.vocab])
    assert e.value.code == ee.EE_EINVAL
    with pytest.raises(ee.EEError) as e:
        eng.extend(0, [1] * 600)          # past max_ctx: nothing committed
    assert e.value.code == ee.EE_ECAPACITY
    assert eng.seq_state(0) == (n0 + 1, nxt)
    eng.close()
