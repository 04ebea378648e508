"""Properties of the GPU path that need no oracle: greedy speculative output
equals the GPU's own token-by-token greedy output bit for bit (the lossless
property of greedy verification), and a row's logits do not depend on how
many rows share its block."""

import numpy as np
import pytest

from workloads import gen_weights, get_shape, planted_draft, zipf_tokens

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ee():
    import paper_2506_02780_amd as mod
    return mod


def _greedy_stream(eng, steps):
    out = []
    for _ in range(steps):
        _, nxt, _ = eng.verify(0, [])
        out.append(nxt)
    return out


@pytest.mark.parametrize("cfg", ["tiny", "bf16"])
def test_speculative_stream_equals_greedy_loop_bitwise(ee, cfg):
    if cfg == "tiny":
        shape, std, k = get_shape("tiny"), 0.1, 8
    else:
        shape = get_shape("tiny", n_layers=2, d_model=512, n_heads=4, n_kv_heads=2, head_dim=128,
                          ffn=1024, vocab=2048, dtype="bf16")
        std, k = 0.05, 32
    w = gen_weights(shape, seed=5, std=std)
    prompt = zipf_tokens(shape.vocab, 70, seed=1)
    eng = ee.Engine(shape, w, max_ctx=512, k_max=k)
    first = eng.prefill(0, prompt)
    target = [first] + _greedy_stream(eng, 120)
    eng.rollback(0, 0, -1)
    assert eng.prefill(0, prompt) == first
    out = [first]
    g = np.random.default_rng(2)
    while len(out) < 100:
        kk = int(g.integers(0, k + 1))
        j = int(g.integers(0, kk + 1))
        d = planted_draft(target[len(out):], j, kk, shape.vocab, seed=int(g.integers(1 << 30)))
        a, nxt, _ = eng.verify(0, d)
        assert a >= j          # planted prefix always accepted
        out += list(d[:a]) + [nxt]
    assert out == target[:len(out)]
    eng.close()


def test_row_logits_independent_of_block_size(ee):
    shape = get_shape("tiny", n_layers=2, d_model=512, n_heads=4, n_kv_heads=2, head_dim=128,
                      ffn=1024, vocab=2048, dtype="bf16")
    w = gen_weights(shape, seed=6, std=0.05)
    prompt = zipf_tokens(shape.vocab, 130, seed=2)
    eng = ee.Engine(shape, w, max_ctx=512, k_max=64)
    first = eng.prefill(0, prompt)
    n0 = eng.seq_state(0)[0]
    ar_rows = []
    toks = [first]
    for _ in range(40):
        _, nxt, _ = eng.verify(0, [])
        ar_rows.append(eng.logits()[0].copy())
        toks.append(nxt)
    for k in (8, 16, 39):
        eng.rollback(0, n0, first)
        a, nxt, _ = eng.verify(0, toks[1:k + 1])
        assert a == k and nxt == toks[k + 1]
        np.testing.assert_array_equal(eng.logits(), np.stack(ar_rows[:k + 1]))
    eng.close()


def test_graph_replays_equal_eager_launches(ee):
    """Every replay of a captured block graph gives the eager result bitwise,
    with eager work and synchronisations between the replays."""
    import torch
    shape = get_shape("tiny", n_layers=2, d_model=512, n_heads=4, n_kv_heads=2, head_dim=128,
                      ffn=1024, vocab=2048, dtype="bf16")
    w = gen_weights(shape, seed=8, std=0.05)
    prompt = zipf_tokens(shape.vocab, 100, seed=3)
    draft = zipf_tokens(shape.vocab, 20, seed=4)
    eng = ee.Engine(shape, w, max_ctx=512, k_max=32)
    first = eng.prefill(0, prompt)
    n0 = eng.seq_state(0)[0]
    eng.use_graphs(False)
    ref = eng.verify(0, draft)
    ref_logits = eng.logits()
    eng.use_graphs(True)
    for rep in range(4):
        eng.rollback(0, n0, first)
        x = torch.randn(1 << 20, device="cuda") * 2.0      # unrelated eager work
        torch.cuda.synchronize()
        got = eng.verify(0, draft)
        assert got[:2] == ref[:2]
        np.testing.assert_array_equal(eng.logits(), ref_logits)
        del x
    eng.close()


def test_graphs_per_split_count_equal_eager_launches(ee):
    """The attention grid covers the splits of the block's context (256
    positions each), so a block shape is captured once per split count:
    contexts on both sides of split boundaries give, from their graphs, the
    eager result bitwise, also when a shape is replayed after others."""
    shape = get_shape("tiny", n_layers=2, d_model=512, n_heads=4, n_kv_heads=2, head_dim=128,
                      ffn=1024, vocab=2048, dtype="bf16")
    w = gen_weights(shape, seed=9, std=0.05)
    prompt = zipf_tokens(shape.vocab, 700, seed=5)
    draft = zipf_tokens(shape.vocab, 20, seed=6)
    eng = ee.Engine(shape, w, max_ctx=1024, k_max=32)
    ctxs = (100, 235, 236, 511, 600)   # n + 21 rows: 1, 1, 2, 3, 3 splits

    def at(n):
        # the prompt's first n tokens committed, its next token pending
        eng.rollback(0, 0, -1)
        eng.prefill(0, prompt)
        eng.rollback(0, n, int(prompt[n]))

    ref = {}
    eng.use_graphs(False)
    for n in ctxs:
        at(n)
        ref[n] = (eng.verify(0, draft)[:2], eng.logits())
    eng.use_graphs(True)
    for n in ctxs + ctxs[::-1]:
        at(n)
        assert eng.verify(0, draft)[:2] == ref[n][0]
        np.testing.assert_array_equal(eng.logits(), ref[n][1])
    eng.close()
