"""Verification at the edges of the paged cache, on the GPU through the C ABI.

Blocks whose committed length n sits at or next to a page boundary (64
positions), an attention split boundary (256), the start of the cache, and
a block that fills the pool to exactly max_ctx (n + K + 1 = max_ctx), for a
linear draft (K = 0 included: one plain greedy step, Eq. 1) and for a draft
tree (the greedy walk).  Each is compared with the oracle on a tiny fp32
model: every logit within 1e-4, the outcome exactly (or, at a near tie, a
correct greedy one) and every committed K/V row within 2e-5.
"""

import numpy as np
import pytest

from oracle import OracleSession
from tests.helpers import valid_outcome
from workloads import gen_weights, get_shape, planted_draft, random_tree, tree_tokens, zipf_tokens

pytestmark = pytest.mark.gpu

MAX_CTX, K_MAX, TOL = 320, 16, 1e-4

# (committed length n, draft length K)
LINEAR = [(1, 0), (1, K_MAX), (2, 5), (63, 0), (63, 1), (64, K_MAX), (127, 7), (192, K_MAX),
          (240, K_MAX), (255, 0), (255, 1), (256, K_MAX), (MAX_CTX - K_MAX - 1, K_MAX), (MAX_CTX - 1, 0)]
# (committed length n, tree nodes)
TREES = [(1, K_MAX), (250, K_MAX), (MAX_CTX - K_MAX - 1, K_MAX)]


@pytest.fixture(scope="module")
def ee():
    import paper_2506_02780_amd as mod
    return mod


@pytest.fixture(scope="module")
def setup(ee):
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=606, std=0.1)
    prompt = zipf_tokens(shape.vocab, MAX_CTX, seed=61)
    eng = ee.Engine(shape, w, max_ctx=MAX_CTX, k_max=K_MAX)
    yield shape, w, prompt, eng
    eng.close()


def _start(shape, w, prompt, eng, n):
    """Both sides with the first n prompt tokens committed and the same token
    pending (the GPU's, if a near tie decided the prefill's last row)."""
    eng.rollback(0, 0, -1)
    ref = OracleSession(shape, w)
    p_ref = ref.prefill(prompt[:n])
    p_gpu = eng.prefill(0, prompt[:n])
    if p_gpu != p_ref:
        err = float(np.abs(eng.logits() - ref.last_logits[-1:]).max())
        assert valid_outcome(ref.last_logits[-1:], [], 0, p_gpu, err)
        ref.pending = p_gpu
    assert eng.seq_state(0) == (n, ref.pending)
    return ref


def _check_cache(shape, eng, ref):
    n = ref.n
    assert eng.seq_state(0) == (n, ref.pending)
    for l in range(shape.n_layers):
        k, v = eng.read_kv(0, l)
        assert k.shape[0] == n
        np.testing.assert_allclose(k, ref.cache[l][0], rtol=0, atol=2e-5)
        np.testing.assert_allclose(v, ref.cache[l][1], rtol=0, atol=2e-5)


@pytest.mark.parametrize("n,k", LINEAR)
def test_linear_block_at_cache_edges_matches_oracle(ee, setup, n, k):
    shape, w, prompt, eng = setup
    ref = _start(shape, w, prompt, eng, n)
    probe = OracleSession(shape, w)
    probe.set_cache(ref.cache, ref.pending)
    truth = probe.greedy(k + 1)
    j = (n * 7 + k) % (k + 1)   # accepted prefix length the draft is planted for
    d = planted_draft(truth, j, k, shape.vocab, seed=n + 13 * k)
    ra, rn, _ = ref.verify(d)
    a, nxt, _ = eng.verify(0, d)
    lg = eng.logits()
    assert lg.shape == (k + 1, shape.vocab)
    err = float(np.abs(lg - ref.last_logits).max())
    assert err <= TOL, f"n={n} K={k}: max |logit difference| {err} > {TOL}"
    if (a, nxt) != (ra, rn):
        assert valid_outcome(ref.last_logits, d, a, nxt, err)
    else:
        assert a == j or k == 0
        _check_cache(shape, eng, ref)
    assert n + a + 1 <= MAX_CTX


@pytest.mark.parametrize("n,k", TREES)
def test_tree_block_at_cache_edges_matches_oracle(ee, setup, n, k):
    shape, w, prompt, eng = setup
    ref = _start(shape, w, prompt, eng, n)
    probe = OracleSession(shape, w)
    probe.set_cache(ref.cache, ref.pending)
    truth = probe.greedy(6)
    parent = random_tree(k, max_depth=5, max_branch=3, seed=n)
    toks = tree_tokens(parent, truth[: 1 + n % 5], shape.vocab, seed=n + 1)
    ra, rn, rpath = ref.verify(toks, parent)
    a, nxt, nodes = eng.verify(0, toks, parent)
    lg = eng.logits()
    err = float(np.abs(lg - ref.last_logits).max())
    assert err <= TOL, f"n={n} tree of {k}: max |logit difference| {err} > {TOL}"
    if (a, nxt, [int(x) + 1 for x in nodes]) == (ra, rn, list(rpath)):
        _check_cache(shape, eng, ref)
    else:
        margins = np.sort(ref.last_logits, axis=1)
        assert float((margins[:, -1] - margins[:, -2])[[0] + list(rpath)].min()) <= 2 * err


def test_full_pool_refuses_one_row_more(ee, setup):
    """A block one row past max_ctx is refused and leaves the state as it was."""
    shape, w, prompt, eng = setup
    n = MAX_CTX - K_MAX
    eng.rollback(0, 0, -1)
    p = eng.prefill(0, prompt[:n])
    with pytest.raises(ee.EEError) as e:
        eng.verify(0, list(prompt[n:n + K_MAX]))   # n + K_MAX + 1 > MAX_CTX
    assert e.value.code == ee.EE_ECAPACITY
    assert eng.seq_state(0) == (n, p)
    a, nxt, _ = eng.verify(0, list(prompt[n:n + K_MAX - 1]))   # exactly full
    assert eng.seq_state(0) == (n + a + 1, nxt)
