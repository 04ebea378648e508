"""Pins of the oracle's whole forward and decoding session (CPU only).

* The forward equals Hugging Face's LlamaForCausalLM (an independent
  implementation of the same decoder) run in float64 on the same weights.
* The KV-cache path equals a full recompute of the whole sequence.
* Speculative greedy verification reproduces plain greedy decoding (the
  lossless property of greedy verification, Sec. "Reuse": tokens are accepted
  only while they equal the target's greedy output).
"""

import numpy as np
import pytest
import torch

from oracle import (OracleSession, accept_linear, accept_tree, chain_structure,
                    forward_block, greedy_rows, tree_structure)
from oracle.numerics import round_bf16, to_f64
from workloads import gen_weights, get_shape, planted_draft, random_tree, zipf_tokens


class _F32View:
    """The same weights widened to fp32 arrays (for an unrounded forward)."""

    def __init__(self, w, dtype):
        self.embed = to_f64(w.embed, dtype).astype(np.float32)
        self.lm_head = to_f64(w.lm_head, dtype).astype(np.float32)
        self.final_gain = w.final_gain
        self._w, self._dt = w, dtype

    def layer(self, l):
        lw = self._w.layer(l)
        return {k: (to_f64(v, self._dt).astype(np.float32) if k.startswith("w") else v)
                for k, v in lw.items()}


def _small(dtype="f32", **kw):
    base = dict(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn=96, vocab=97)
    base.update(kw)
    return get_shape("tiny", dtype=dtype, **base)


def _hf_logits(shape, w, tokens):
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = LlamaConfig(vocab_size=shape.vocab, hidden_size=shape.d_model,
                      intermediate_size=shape.ffn, num_hidden_layers=shape.n_layers,
                      num_attention_heads=shape.n_heads, num_key_value_heads=shape.n_kv_heads,
                      head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
                      rope_theta=shape.rope_theta, tie_word_embeddings=False,
                      max_position_embeddings=4096, attention_bias=False, mlp_bias=False)
    m = LlamaForCausalLM(cfg).double().eval()
    sd = {"model.embed_tokens.weight": w.embed, "lm_head.weight": w.lm_head,
          "model.norm.weight": w.final_gain}
    names = {"wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "w_gate": "mlp.gate_proj", "w_up": "mlp.up_proj",
             "w_down": "mlp.down_proj", "attn_gain": "input_layernorm",
             "ffn_gain": "post_attention_layernorm"}
    for l in range(shape.n_layers):
        for k, v in w.layer(l).items():
            sd[f"model.layers.{l}.{names[k]}.weight"] = v
    m.load_state_dict({k: torch.from_numpy(np.asarray(v, dtype=np.float64)) for k, v in sd.items()},
                      strict=True)
    with torch.no_grad():
        return m(torch.tensor(np.asarray(tokens)[None, :], dtype=torch.long)).logits[0].numpy()


@pytest.mark.slow
def test_forward_matches_hf_llama():
    shape = _small()
    w = gen_weights(shape, seed=3, gains="random", std=0.1)
    toks = zipf_tokens(shape.vocab, 40, seed=1)
    sess = OracleSession(shape, w)
    sess.prefill(toks)
    ref = _hf_logits(shape, w, toks)
    # HF evaluates RoPE angles and RMSNorm in fp32 even in a float64 model
    np.testing.assert_allclose(sess.last_logits, ref, rtol=0, atol=2e-5)
    assert np.abs(ref).max() > 0.5


def test_incremental_cache_equals_full_recompute():
    shape = _small()
    w = gen_weights(shape, seed=4, gains="random", std=0.1)
    toks = zipf_tokens(shape.vocab, 30, seed=2)
    full_depth, full_vis = chain_structure(30)
    full, _ = forward_block(shape, w, [], toks, full_depth, full_vis)
    sess = OracleSession(shape, w)
    sess.prefill(toks[:11])
    np.testing.assert_allclose(sess.last_logits, full[:11], rtol=0, atol=1e-12)
    # feed the true continuation as a draft: every row must reproduce full[]
    sess.rollback(11, int(toks[11]))
    a, nxt, _ = sess.verify(toks[12:20])
    np.testing.assert_allclose(sess.last_logits, full[11:20], rtol=0, atol=1e-12)
    assert sess.n == 12 + a
    # roll back below the prompt and continue from there
    sess.rollback(5, int(toks[5]))
    sess.verify(toks[6:30])
    np.testing.assert_allclose(sess.last_logits, full[5:30], rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_speculative_greedy_equals_plain_greedy(seed):
    shape = _small()
    w = gen_weights(shape, seed=100 + seed, std=0.1)
    prompt = zipf_tokens(shape.vocab, 12, seed=seed)
    ref = OracleSession(shape, w)
    ref.prefill(prompt)
    target = [ref.pending] + ref.greedy(60)
    spec = OracleSession(shape, w)
    spec.prefill(prompt)
    out = [spec.pending]
    g = np.random.default_rng(seed)
    while len(out) < 40:
        k = int(g.integers(0, 9))
        j = int(g.integers(0, k + 1))
        true_next = target[len(out):]
        d = planted_draft(true_next, j, k, shape.vocab, seed=int(g.integers(1 << 30)))
        a, nxt, _ = spec.verify(d)
        assert a == j
        out += list(d[:a]) + [nxt]
    assert out == target[:len(out)]


def test_planted_draft_accepts_exactly_j():
    shape = _small()
    w = gen_weights(shape, seed=7, std=0.1)
    base = OracleSession(shape, w)
    base.prefill(zipf_tokens(shape.vocab, 10, seed=3))
    probe = OracleSession(shape, w)
    probe.set_cache([(k, v) for k, v in base.cache], base.pending)
    true_next = probe.greedy(8)
    for j in range(9):
        s = OracleSession(shape, w)
        s.set_cache([(k, v) for k, v in base.cache], base.pending)
        d = planted_draft(true_next, j, 8, shape.vocab, seed=j)
        a, nxt, _ = s.verify(d)
        assert a == j
        assert nxt == true_next[j] if j < 8 else True
        assert s.n == base.n + 1 + j


def test_accept_linear_closed_form():
    g = np.random.default_rng(9)
    for _ in range(500):
        k = int(g.integers(0, 12))
        gr = g.integers(0, 3, k + 1)
        d = g.integers(0, 3, k)
        mism = np.nonzero(d != gr[:k])[0]
        a_ref = int(mism[0]) if len(mism) else k
        assert accept_linear(d, gr) == (a_ref, int(gr[a_ref]))


def test_chain_shaped_tree_equals_linear():
    shape = _small()
    w = gen_weights(shape, seed=8, std=0.1)
    prompt = zipf_tokens(shape.vocab, 9, seed=4)
    d = zipf_tokens(shape.vocab, 6, seed=5)
    s1, s2 = OracleSession(shape, w), OracleSession(shape, w)
    s1.prefill(prompt)
    s2.prefill(prompt)
    r1 = s1.verify(d)
    r2 = s2.verify(d, parent=np.arange(-1, 5))
    np.testing.assert_array_equal(s1.last_logits, s2.last_logits)
    assert r1[:2] == r2[:2]


def test_tree_rows_equal_linear_rows_of_their_path_and_walk_is_best_path():
    shape = _small()
    w = gen_weights(shape, seed=9, std=0.1)
    base = OracleSession(shape, w)
    base.prefill(zipf_tokens(shape.vocab, 7, seed=6))
    cache = [(k, v) for k, v in base.cache]
    probe = OracleSession(shape, w)
    probe.set_cache(cache, base.pending)
    greedy_chain = probe.greedy(6)
    parent = random_tree(16, max_depth=5, max_branch=3, seed=3)
    from workloads import tree_tokens
    tok = tree_tokens(parent, greedy_chain, shape.vocab, seed=3)
    t = OracleSession(shape, w)
    t.set_cache(cache, base.pending)
    a, nxt, path = t.verify(tok, parent=parent)
    tree_logits = t.last_logits
    depth, vis = tree_structure(parent)
    best = -1
    for r in range(1, len(tok) + 1):
        anc = [c for c in range(1, r + 1) if vis[r, c]]          # depth order
        lin = OracleSession(shape, w)
        lin.set_cache(cache, base.pending)
        la, _, _ = lin.verify(tok[np.array(anc) - 1])
        np.testing.assert_allclose(tree_logits[r], lin.last_logits[-1], rtol=0, atol=1e-11)
        # a leaf's path accepts la tokens along it
        if not any(parent[i] + 1 == r for i in range(len(tok))):
            best = max(best, la)
    assert a == best
    assert a == len(path) and t.n == base.n + 1 + a


def test_bf16_mode_rounds_cache_and_stays_near_unrounded():
    shape = _small(dtype="bf16")
    w = gen_weights(shape, seed=10, std=0.1)
    toks = zipf_tokens(shape.vocab, 20, seed=7)
    s = OracleSession(shape, w)
    s.prefill(toks)
    for k, v in s.cache:
        np.testing.assert_array_equal(round_bf16(k), k)
        np.testing.assert_array_equal(round_bf16(v), v)
    exact = OracleSession(shape.with_(dtype="f32"), _F32View(w, "bf16"))
    exact.prefill(toks)
    diff = np.abs(s.last_logits - exact.last_logits).max()
    # every bf16 rounding perturbs by at most 2^-9 relative
    assert 0 < diff < 0.02 * np.abs(exact.last_logits).max()


def test_rounding_hook_is_off_by_default_and_only_sees_bf16_sites():
    """The rounding-site hook leaves the definition alone: a hook that returns
    the definition's rounding gives the same forward bit for bit, an fp32
    model has no rounding sites for it to see, and on a bf16 model the noise
    probe with a float32-sized error moves the logits a little (an operand
    within that error of a rounding boundary rounds the other way) and a
    larger error more."""
    from tests.helpers import noise_probe
    toks = zipf_tokens(97, 24, seed=3)
    depth, vis = chain_structure(len(toks))
    for dt in ("f32", "bf16"):
        shape = _small(dt)
        w = gen_weights(shape, seed=4, std=0.2)
        exact, _ = forward_block(shape, w, [], toks, depth, vis)
        seen = []
        same, _ = forward_block(shape, w, [], toks, depth, vis,
                                rounding=lambda s, l, e, r: (seen.append((s, l)), r)[1])
        assert np.array_equal(exact, same)
        tiny, _ = forward_block(shape, w, [], toks, depth, vis, noise_probe(np.random.default_rng(1), 2.0 ** -23))
        big, _ = forward_block(shape, w, [], toks, depth, vis, noise_probe(np.random.default_rng(1), 2.0 ** -12))
        if dt == "f32":
            assert seen == []
            assert np.array_equal(exact, tiny) and np.array_equal(exact, big)
        else:
            assert len(seen) == 7 * shape.n_layers + 1
            d_tiny = np.abs(tiny - exact).max()
            d_big = np.abs(big - exact).max()
            assert d_tiny < 0.05 * np.abs(exact).max()
            assert d_tiny < d_big
