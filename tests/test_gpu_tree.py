"""Tree-structured drafts on the GPU, through the C ABI.

* parity with the oracle: every row's logits, the greedy tree walk and the KV
  cache after compaction;
* a tree row is bit-identical to the same token path verified as a linear
  chain (its ancestors sit at the positions the chain would give them), so
  the committed cache and the emitted stream are those of plain greedy
  decoding, bit for bit.
"""

import numpy as np
import pytest

from oracle import OracleSession, top2_margin
from oracle.accept import accept_tree
from oracle.numerics import to_f64
from workloads import gen_weights, get_shape, random_tree, tree_tokens, zipf_tokens

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


def _tree(step, k, max_depth, branch, truth, vocab, seed):
    """A random tree whose first-child chain follows the true continuation for
    a random number of levels, then diverges."""
    g = np.random.default_rng(seed + step)
    if max_depth <= 12:
        parent = random_tree(k, max_depth=max_depth, max_branch=branch, seed=seed + 31 * step)
    else:
        # deep tree: a spine of max_depth nodes, the rest hung on random earlier nodes
        parent = np.arange(-1, k - 1, dtype=np.int32)
        for i in range(max_depth, k):
            parent[i] = int(g.integers(-1, i))
    j = int(g.integers(0, max_depth + 1))
    toks = tree_tokens(parent, truth[:j], vocab, seed=seed + 7 * step)
    return parent, toks


def _path_rows(parent, node):
    """Block rows from the pending row down to `node` (a node index)."""
    rows = []
    while node >= 0:
        rows.append(node + 1)
        node = int(parent[node])
    return [0] + rows[::-1]


@pytest.mark.parametrize("cfg", ["tiny", "bf16", "bf16_g4"])
def test_tree_verify_matches_oracle(ee, cfg):
    if cfg == "tiny":
        shape, tol, std = get_shape("tiny"), 1e-4, 0.1
    elif cfg == "bf16":
        shape, tol, std = _bf16_small(), 2e-2, 0.02
    else:
        # 4 query heads per KV head: 64-node trees take the two-launch path
        shape, tol, std = _bf16_small(d_model=1024, n_heads=8), 2e-2, 0.02
    w = gen_weights(shape, seed=41, std=std, gains="random")
    prompt = zipf_tokens(shape.vocab, 237, seed=12)     # blocks cross a 256-position split
    ref = OracleSession(shape, w)
    ref.prefill(prompt)
    eng = ee.Engine(shape, w, max_ctx=640, k_max=64)
    eng.prefill(0, prompt)
    shapes = [(64, 8, 3), (48, 40, 2), (20, 6, 3), (64, 8, 3), (40, 30, 2), (64, 8, 3)]
    pinned = 0
    for step, (k, depth, branch) in enumerate(shapes):
        n_before, p_before = ref.n, ref.pending
        probe = OracleSession(shape, w)
        probe.set_cache(ref.cache, ref.pending)
        truth = probe.greedy(depth)
        parent, toks = _tree(step, k, depth, branch, truth, shape.vocab, seed=100)
        ra, rn, rpath = ref.verify(toks, parent)
        a, n, nodes = eng.verify(0, toks, parent)
        lg = eng.logits()
        err = float(np.abs(lg - ref.last_logits).max())
        assert err <= tol, f"step {step}: max |logit difference| {err} > {tol}"
        # the GPU's walk is exactly the greedy walk over its own logits (lowest
        # index on ties), at every step
        ga, gn, gpath = accept_tree(toks, parent, np.argmax(lg, axis=1))
        assert (a, n, [int(x) + 1 for x in nodes]) == (ga, gn, gpath), f"step {step}: walk"
        same = (a, n) == (ra, rn) and [int(x) + 1 for x in nodes] == list(rpath)
        deciding = float(top2_margin(ref.last_logits)[[0] + list(rpath)].min())
        if not same:
            # only a near tie on the walk may decide the other way; both sides
            # then return to the state before the step
            assert deciding <= tol, f"step {step}: outcome differs at top-2 margin {deciding}"
            ref.rollback(n_before, p_before)
            eng.rollback(0, n_before, p_before)
            continue
        assert eng.seq_state(0) == (ref.n, ref.pending)
        pinned += 1
    assert pinned >= 2
    for l in range(shape.n_layers):
        k_, v_ = eng.read_kv(0, l)
        rk, rv = ref.cache[l]
        kk, vv = to_f64(k_, shape.dtype), to_f64(v_, shape.dtype)
        scale = max(1.0, float(np.abs(rk).max()))
        assert np.abs(kk - rk).max() <= (2e-5 if cfg == "tiny" else 2e-2) * scale
        assert np.abs(vv - rv).max() <= (2e-5 if cfg == "tiny" else 2e-2) * scale
    eng.close()


@pytest.mark.parametrize("prompt_len,heads", [(150, 4), (250, 4), (150, 8), (255, 8), (300, 8)])
def test_tree_rows_equal_chain_rows_bitwise(ee, prompt_len, heads):
    # heads = 8 (4 query heads per KV head): the 64-node tree has 17 query
    # tiles and runs the wide kernel's work over the splits below its rows and
    # the tree kernel's over the splits holding them, in one launch (from slot
    # n + 1: split 0 at n = 150, split 1 at n = 255 and 300); the 40-node tree
    # runs the tree kernel alone
    shape = _bf16_small() if heads == 4 else _bf16_small(d_model=1024, n_heads=8)
    w = gen_weights(shape, seed=42, std=0.05)
    prompt = zipf_tokens(shape.vocab, prompt_len, seed=13)
    eng = ee.Engine(shape, w, max_ctx=640, k_max=64)
    first = eng.prefill(0, prompt)
    n0 = eng.seq_state(0)[0]
    truth = []
    for _ in range(12):
        truth.append(eng.verify(0, [])[1])
    for step, (k, depth, branch) in enumerate([(64, 8, 3), (40, 30, 2)]):
        eng.rollback(0, n0, first)
        parent, toks = _tree(step, k, depth, branch, truth, shape.vocab, seed=200)
        a, nxt, nodes = eng.verify(0, toks, parent)
        tree_lg = eng.logits()
        tree_kv = [eng.read_kv(0, l) for l in range(shape.n_layers)]
        leaves = sorted(set(range(k)) - set(int(p) for p in parent))
        g = np.random.default_rng(step)
        chosen = [int(nodes[-1]) if a else None] + [int(x) for x in g.choice(leaves, 3, replace=False)]
        for leaf in chosen:
            rows = [0] if leaf is None else _path_rows(parent, leaf)
            eng.rollback(0, n0, first)
            ca, cn, _ = eng.verify(0, toks[np.asarray(rows[1:], dtype=np.int64) - 1])
            np.testing.assert_array_equal(eng.logits(), tree_lg[rows])
            if leaf == (int(nodes[-1]) if a else None):
                # the accepted path: same outcome and the same committed cache
                assert (ca, cn) == (a, nxt)
                for l in range(shape.n_layers):
                    ck, cv = eng.read_kv(0, l)
                    np.testing.assert_array_equal(ck, tree_kv[l][0])
                    np.testing.assert_array_equal(cv, tree_kv[l][1])
    eng.close()


@pytest.mark.parametrize("cfg", ["tiny", "bf16"])
def test_tree_stream_equals_greedy_loop_bitwise(ee, cfg):
    if cfg == "tiny":
        shape, std = get_shape("tiny"), 0.1
    else:
        shape, std = _bf16_small(), 0.05
    w = gen_weights(shape, seed=43, std=std)
    prompt = zipf_tokens(shape.vocab, 190, seed=14)
    eng = ee.Engine(shape, w, max_ctx=640, k_max=64)
    first = eng.prefill(0, prompt)
    target = [first] + [eng.verify(0, [])[1] for _ in range(150)]
    eng.rollback(0, 0, -1)
    assert eng.prefill(0, prompt) == first
    out = [first]
    step = 0
    while len(out) < 120:
        k, depth, branch = [(64, 8, 3), (30, 12, 2), (10, 4, 3)][step % 3]
        parent, toks = _tree(step, k, depth, branch, target[len(out):], shape.vocab, seed=300)
        a, nxt, nodes = eng.verify(0, toks, parent)
        out += [int(toks[i]) for i in nodes] + [nxt]
        step += 1
    assert out == target[:len(out)]
    eng.close()
