"""ee_verify_noalloc, the allocation-free variant of ee_verify, against
ee_verify itself through the C ABI: two calls in a row (the second with a
smaller block) give the same accept length, next token, logits and committed
K/V bit for bit, for a linear draft and a draft tree; a block whose scratch
would exceed the static 16 MiB array is refused before it runs and leaves
the sequence unchanged."""

import numpy as np
import pytest

from workloads import gen_weights, get_shape, planted_draft, random_tree, tree_tokens, zipf_tokens

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ee():
    import paper_2506_02780_amd as mod
    return mod


def _same_step(eng, n0, p0, draft, parent=None):
    eng.rollback(0, n0, p0)
    ra = eng.verify(0, draft, parent)
    rl = eng.logits()
    rk, rv = eng.read_kv(0, 0)
    rs = eng.seq_state(0)
    eng.rollback(0, n0, p0)
    ga = eng.verify_noalloc(0, draft, parent)
    gl = eng.logits()
    gk, gv = eng.read_kv(0, 0)
    assert ga[:2] == ra[:2]
    if parent is not None:
        assert np.array_equal(ga[2], ra[2])
    assert np.array_equal(gl, rl)
    assert eng.seq_state(0) == rs
    assert np.array_equal(gk, rk) and np.array_equal(gv, rv)
    return ga


def test_noalloc_equals_verify_bf16_two_calls(ee):
    shape = get_shape("tiny", n_layers=2, d_model=512, n_heads=8, n_kv_heads=2, head_dim=128, ffn=1024,
                      vocab=2048, dtype="bf16")
    w = gen_weights(shape, seed=61, std=0.05)
    eng = ee.Engine(shape, w, max_ctx=640, k_max=64)
    prompt = zipf_tokens(shape.vocab, 300, seed=62)
    first = eng.prefill(0, prompt)
    n0 = eng.seq_state(0)[0]
    cont = [first] + [eng.verify(0, [])[1] for _ in range(40)]
    eng.rollback(0, n0, first)
    # first call: 41 rows, 20 of the draft accepted; second: a smaller block
    a1 = _same_step(eng, n0, first, planted_draft(cont[1:], 20, 40, shape.vocab, seed=1))
    assert a1[0] == 20
    a2 = _same_step(eng, n0, first, planted_draft(cont[1:], 3, 6, shape.vocab, seed=2))
    assert a2[0] == 3
    parent = random_tree(24, max_depth=5, max_branch=3, seed=4)
    _same_step(eng, n0, first, tree_tokens(parent, cont[1:6], shape.vocab, seed=4), parent)
    eng.close()


def test_noalloc_equals_verify_fp32_two_calls(ee):
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=63, std=0.1)
    eng = ee.Engine(shape, w, max_ctx=512, k_max=32)
    first = eng.prefill(0, zipf_tokens(shape.vocab, 100, seed=64))
    n0 = eng.seq_state(0)[0]
    d = zipf_tokens(shape.vocab, 16, seed=65)
    _same_step(eng, n0, first, d)
    _same_step(eng, n0, first, d[:5])
    eng.close()


def test_noalloc_refuses_blocks_beyond_its_static_scratch(ee):
    """A 513-row block over 2000 committed positions of a bf16 model with
    head_dim 128 and 4 query heads per KV head needs ~25 MB of scratch (10
    attention splits of 2 KV heads x 2052 query columns x 130 floats, plus
    the LM head's partials): refused before it runs, the sequence unchanged;
    a small block on the same sequence still runs."""
    shape = get_shape("tiny", n_layers=1, d_model=512, n_heads=8, n_kv_heads=2, head_dim=128, ffn=1024,
                      vocab=2048, dtype="bf16")
    w = gen_weights(shape, seed=66, std=0.05)
    eng = ee.Engine(shape, w, max_ctx=2600, k_max=512)
    eng.prefill(0, zipf_tokens(shape.vocab, 2000, seed=67))
    st = eng.seq_state(0)
    with pytest.raises(ee.EEError) as e:
        eng.verify_noalloc(0, zipf_tokens(shape.vocab, 512, seed=68))
    assert e.value.code == ee.EE_ECAPACITY and "16 MiB" in str(e.value)
    assert eng.seq_state(0) == st
    _same_step(eng, st[0], st[1], zipf_tokens(shape.vocab, 8, seed=69))
    eng.close()
