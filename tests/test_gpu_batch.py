"""Several sequences verified in one block (ee_verify_batch), through the C ABI.

Each sequence reads only its own paged cache and its rows are computed with
the same arithmetic as in a block of its own, so batched results must equal
single-sequence results bit for bit; against the oracle they are held to
the usual tolerances.
"""

import numpy as np
import pytest

from oracle import OracleSession
from tests.helpers import assert_step_matches, reuse_draft
from workloads import gen_weights, get_shape, planted_draft, random_tree, tree_tokens, zipf_tokens

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


def _engine(ee, shape, w, prompts, k_max=64, max_ctx=640):
    eng = ee.Engine(shape, w, max_ctx=max_ctx, max_seqs=len(prompts), k_max=k_max)
    firsts = [eng.prefill(b, p) for b, p in enumerate(prompts)]
    return eng, firsts


def _continuations(eng, n_seq, steps):
    """Each sequence's own greedy continuation (single-sequence K = 0 steps),
    rolled back afterwards."""
    out = []
    for b in range(n_seq):
        n0, p0 = eng.seq_state(b)
        out.append([eng.verify(b, [])[1] for _ in range(steps)])
        eng.rollback(b, n0, p0)
    return out


@pytest.mark.parametrize("tree", [False, True])
def test_batch_rows_equal_single_sequence_rows_bitwise(ee, tree):
    shape = _bf16_small()
    w = gen_weights(shape, seed=51, std=0.05)
    prompts = [zipf_tokens(shape.vocab, n, seed=60 + i) for i, n in enumerate((100, 190, 250, 301))]
    eng, _ = _engine(ee, shape, w, prompts)
    B, K = 4, 64
    truth = _continuations(eng, B, 10)
    states = [eng.seq_state(b) for b in range(B)]
    drafts, parents = [], []
    for b in range(B):
        if tree:
            par = random_tree(K, max_depth=8, max_branch=3, seed=70 + b)
            drafts.append(tree_tokens(par, truth[b][:3 + 2 * b], shape.vocab, seed=80 + b))
            parents.append(par)
        else:
            drafts.append(planted_draft(truth[b], 2 * b + 1, K, shape.vocab, seed=90 + b))
    single, single_logits, single_kv = [], [], []
    for b in range(B):
        single.append(eng.verify(b, drafts[b], parents[b] if tree else None))
        single_logits.append(eng.logits())
        single_kv.append([eng.read_kv(b, l) for l in range(shape.n_layers)])
        eng.rollback(b, *states[b])
    res = eng.verify_batch(list(range(B)), drafts, parents if tree else None)
    lg = eng.logits()
    assert lg.shape[0] == B * (K + 1)
    for b in range(B):
        np.testing.assert_array_equal(lg[b * (K + 1):(b + 1) * (K + 1)], single_logits[b])
        assert res[b][:2] == single[b][:2]
        if tree:
            np.testing.assert_array_equal(res[b][2], single[b][2])
        for l in range(shape.n_layers):
            k, v = eng.read_kv(b, l)
            np.testing.assert_array_equal(k, single_kv[b][l][0])
            np.testing.assert_array_equal(v, single_kv[b][l][1])
    eng.close()


def test_batch_reuse_sessions_match_oracle(ee):
    """Three tiny fp32 Reuse sessions advanced together, each against its own
    oracle session."""
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=1234)
    codes = [zipf_tokens(shape.vocab, 192, seed=42 + i) for i in range(3)]
    refs, gens, curs = [], [], []
    for c in codes:
        r = OracleSession(shape, w)
        r.prefill(c[:64 - 8 * len(refs)])
        refs.append(r)
        gens.append([r.pending])
        curs.append(0)
    eng, firsts = _engine(ee, shape, w, [c[:64 - 8 * i] for i, c in enumerate(codes)], k_max=8, max_ctx=320)
    assert firsts == [r.pending for r in refs]
    live = [True] * 3
    for step in range(10):
        drafts, starts = [], []
        for b in range(3):
            st, d = reuse_draft(gens[b], codes[b], curs[b], 8)
            d = np.concatenate([d, zipf_tokens(shape.vocab, 8 - len(d), seed=step)]).astype(np.int32)
            drafts.append(d)
            starts.append(st)
        res = eng.verify_batch([0, 1, 2], drafts)
        lg = eng.logits()
        for b in range(3):
            if not live[b]:
                continue
            ra, rn, _ = refs[b].verify(drafts[b])
            same = assert_step_matches(lg[b * 9:(b + 1) * 9], res[b][0], res[b][1], refs[b].last_logits,
                                       ra, rn, 8, 1e-4)
            if not same:
                live[b] = False
                continue
            gens[b] += list(drafts[b][:ra]) + [rn]
            curs[b] = starts[b] + ra + 1
            assert eng.seq_state(b) == (refs[b].n, refs[b].pending)
    assert all(live)
    eng.close()


def test_batch_streams_equal_each_greedy_loop_bitwise(ee):
    shape = _bf16_small()
    w = gen_weights(shape, seed=52, std=0.05)
    prompts = [zipf_tokens(shape.vocab, n, seed=100 + i) for i, n in enumerate((120, 77, 260))]
    eng, firsts = _engine(ee, shape, w, prompts)
    target = _continuations(eng, 3, 160)
    outs = [[] for _ in range(3)]
    g = np.random.default_rng(3)
    K = 16
    while min(len(o) for o in outs) < 80:
        drafts = []
        for b in range(3):
            rest = target[b][len(outs[b]):]
            j = min(int(g.integers(0, K + 1)), len(rest))
            drafts.append(planted_draft(rest, j, K, shape.vocab, seed=int(g.integers(1 << 30))))
        for b, (a, nxt, _) in enumerate(eng.verify_batch([0, 1, 2], drafts)):
            outs[b] += list(drafts[b][:a]) + [nxt]
    for b in range(3):
        n = min(len(outs[b]), len(target[b]))
        assert outs[b][:n] == target[b][:n]
    eng.close()


def test_batch_errors_leave_every_sequence_unchanged(ee):
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=3)
    prompts = [zipf_tokens(shape.vocab, n, seed=7 + n) for n in (40, 190)]
    eng, _ = _engine(ee, shape, w, prompts, k_max=16, max_ctx=200)
    before = [eng.seq_state(b) for b in range(2)]
    d = [list(range(1, 11)), list(range(2, 12))]
    with pytest.raises(ee.EEError) as e:
        eng.verify_batch([0, 0], d)                       # a sequence twice
    assert e.value.code == ee.EE_EINVAL
    with pytest.raises(ee.EEError) as e:
        eng.verify_batch([0, 1, 1], d + [d[0]])           # more than max_seqs
    assert e.value.code == ee.EE_EINVAL
    with pytest.raises(ee.EEError) as e:
        eng.verify_batch([0, 1], d)                       # 190 + 11 > 200 for sequence 1
    assert e.value.code == ee.EE_ECAPACITY
    assert [eng.seq_state(b) for b in range(2)] == before
    res = eng.verify_batch([1, 0], [d[0][:5], d[1][:5]])  # fits, in either order
    assert [eng.seq_state(b)[0] for b in range(2)] == [before[0][0] + 1 + res[1][0], before[1][0] + 1 + res[0][0]]
    eng.close()
