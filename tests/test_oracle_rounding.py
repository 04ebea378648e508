"""Pin of the oracle's bf16 rounding sites (CPU only).

The paper states no precision, so where a bf16 pipeline rounds is a reading
(the oracle's ``ROUNDING_SITES``: the inputs of the projections that follow a
norm, taken as h * g; q and k after RoPE; v; the attention output; the SwiGLU
product; the LM head's input).  This test evaluates the same decoder a second,
independent way: Hugging Face's ``LlamaForCausalLM`` in float64, with torch's
own bf16 casts (``Tensor.to(torch.bfloat16)``) applied through module hooks at
exactly those sites.  The oracle must agree with it to float64 rounding
(1e-12), and leaving out the rounding at any single site, or adding one at
the norm's output instead of at h * g, must break that agreement, so the
oracle's list of sites is fixed by something other than the oracle itself.

Hugging Face evaluates the RoPE angles, RMSNorm and softmax in float32 even in
a float64 model; here the angles are computed in float64, the projections'
inputs are built from the norm's input h in float64 (r (h g) with
r = 1 / sqrt(mean h^2 + eps)), and attention runs through torch's scaled dot
product attention in float64.  Everything else (residual wiring, head
grouping, rotate-half pairing, masking, SwiGLU, LM head) is Hugging Face's.
"""

import numpy as np
import pytest
import torch

from oracle import chain_structure, forward_block
from oracle.model import ROUNDING_SITES
from workloads import gen_weights, get_shape, zipf_tokens


def _shape():
    return get_shape("tiny", dtype="bf16", n_layers=2, d_model=64, n_heads=4, n_kv_heads=2,
                     head_dim=16, ffn=96, vocab=97)


def _bf16(t):
    return t.to(torch.bfloat16).to(torch.float64)


def _hf_rounded_logits(shape, w, tokens, skip=None, norm_output_site=False):
    """Logits of HF Llama (float64) with bf16 casts at the rounding sites.
    skip: a site left unrounded.  norm_output_site: round RMSNorm(h) * g
    instead of h * g before the projections (a different reading)."""
    import transformers.models.llama.modeling_llama as ml
    from transformers import LlamaConfig, LlamaForCausalLM

    cfg = LlamaConfig(vocab_size=shape.vocab, hidden_size=shape.d_model, intermediate_size=shape.ffn,
                      num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_heads,
                      num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim,
                      rms_norm_eps=shape.rms_eps, rope_theta=shape.rope_theta, tie_word_embeddings=False,
                      max_position_embeddings=4096, attention_bias=False, mlp_bias=False)
    cfg._attn_implementation = "sdpa"
    m = LlamaForCausalLM(cfg).double().eval()
    from oracle.numerics import to_f64
    sd = {"model.embed_tokens.weight": to_f64(w.embed, "bf16"), "lm_head.weight": to_f64(w.lm_head, "bf16"),
          "model.norm.weight": w.final_gain}
    names = {"wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "w_gate": "mlp.gate_proj", "w_up": "mlp.up_proj",
             "w_down": "mlp.down_proj", "attn_gain": "input_layernorm", "ffn_gain": "post_attention_layernorm"}
    for l in range(shape.n_layers):
        for k, v in w.layer(l).items():
            sd[f"model.layers.{l}.{names[k]}.weight"] = to_f64(v, "bf16") if k.startswith("w") else v
    m.load_state_dict({k: torch.from_numpy(np.asarray(v, dtype=np.float64)) for k, v in sd.items()}, strict=True)

    def rnd(site, t):
        return t if site == skip else _bf16(t)

    # RoPE angles in float64 (HF computes them in float32)
    hd, theta = shape.head_dim, shape.rope_theta
    inv = theta ** (-torch.arange(0, hd, 2, dtype=torch.float64) / hd)

    def rotary(x, position_ids):
        fr = position_ids[..., None].to(torch.float64) * inv
        emb = torch.cat([fr, fr], dim=-1)
        return emb.cos(), emb.sin()

    m.model.rotary_emb.forward = rotary

    hooks, seen = [], {}

    def norm_input(key):
        def pre(mod, args):
            seen[key] = args[0]
        return pre

    def proj_input(key, norm, site):
        def pre(mod, args):
            h = seen[key]
            r = torch.rsqrt((h * h).mean(-1, keepdim=True) + shape.rms_eps)
            if norm_output_site:
                return (rnd(site, h * r * norm.weight),)
            return (rnd(site, h * norm.weight) * r,)
        return pre

    for l, layer in enumerate(m.model.layers):
        at, mlp = layer.self_attn, layer.mlp
        hooks.append(layer.input_layernorm.register_forward_pre_hook(norm_input(("a", l))))
        hooks.append(layer.post_attention_layernorm.register_forward_pre_hook(norm_input(("f", l))))
        for p in (at.q_proj, at.k_proj, at.v_proj):
            hooks.append(p.register_forward_pre_hook(proj_input(("a", l), layer.input_layernorm, "x_attn")))
        for p in (mlp.gate_proj, mlp.up_proj):
            hooks.append(p.register_forward_pre_hook(proj_input(("f", l), layer.post_attention_layernorm, "x_ffn")))
        hooks.append(at.v_proj.register_forward_hook(lambda mod, args, out: rnd("v", out)))
        hooks.append(at.o_proj.register_forward_pre_hook(lambda mod, args: (rnd("o", args[0]),)))
        hooks.append(mlp.down_proj.register_forward_pre_hook(lambda mod, args: (rnd("z", args[0]),)))
    hooks.append(m.model.norm.register_forward_pre_hook(norm_input(("final", 0))))
    hooks.append(m.lm_head.register_forward_pre_hook(proj_input(("final", 0), m.model.norm, "x_final")))

    orig = ml.apply_rotary_pos_emb

    def rope_rounded(q, k, cos, sin, unsqueeze_dim=1):
        qe, ke = orig(q, k, cos, sin, unsqueeze_dim)
        return rnd("q", qe), rnd("k", ke)

    ml.apply_rotary_pos_emb = rope_rounded
    try:
        with torch.no_grad():
            out = m(torch.tensor(np.asarray(tokens)[None, :], dtype=torch.long)).logits[0].numpy()
    finally:
        ml.apply_rotary_pos_emb = orig
        for hk in hooks:
            hk.remove()
    return out


@pytest.fixture(scope="module")
def case():
    shape = _shape()
    w = gen_weights(shape, seed=31, gains="random", std=0.1)
    toks = zipf_tokens(shape.vocab, 24, seed=5)
    depth, vis = chain_structure(len(toks))
    return shape, w, toks, depth, vis


@pytest.mark.slow
def test_oracle_rounding_sites_equal_hf_llama_with_bf16_casts(case):
    shape, w, toks, depth, vis = case
    ref = _hf_rounded_logits(shape, w, toks)
    got, _ = forward_block(shape, w, [], toks, depth, vis)
    assert np.abs(ref).max() > 0.5
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


@pytest.mark.slow
@pytest.mark.parametrize("site", ROUNDING_SITES)
def test_dropping_one_rounding_site_breaks_the_pin(case, site):
    """A planted oracle mistake: one site left unrounded.  The pin above must
    see it (and HF with the same site skipped must agree again, so the site
    names mean the same thing on both sides)."""
    shape, w, toks, depth, vis = case
    ref = _hf_rounded_logits(shape, w, toks)
    skip = lambda s, l, exact, rounded: exact if s == site else rounded
    got, _ = forward_block(shape, w, [], toks, depth, vis, rounding=skip)
    assert np.abs(got - ref).max() > 1e-6, f"dropping the {site} rounding went unnoticed"
    ref_skip = _hf_rounded_logits(shape, w, toks, skip=site)
    np.testing.assert_allclose(got, ref_skip, rtol=0, atol=1e-12)


@pytest.mark.slow
def test_rounding_the_norm_output_instead_of_h_times_g_breaks_the_pin(case):
    """The other natural reading (round RMSNorm(h) * g) is a different model
    at the bf16 level; the pin tells them apart."""
    shape, w, toks, depth, vis = case
    ref_other = _hf_rounded_logits(shape, w, toks, norm_output_site=True)
    got, _ = forward_block(shape, w, [], toks, depth, vis)
    assert np.abs(got - ref_other).max() > 1e-6


def test_rounding_check_accepts_float32_sized_choices_and_rejects_errors(case):
    """The validator the full-width GPU tests use, pinned on the CPU: values
    stored by an evaluation with a float32-sized error at every rounding site
    (the noise probe) are all accepted, the forward that follows them
    reproduces that evaluation's logits, and a value off by two bf16 steps is
    reported as a mismatch."""
    from oracle.numerics import round_bf16
    from tests.helpers import RoundingCheck, noise_probe
    shape, w, toks, depth, vis = case
    stored = {}
    probe = noise_probe(np.random.default_rng(3), 2.0 ** -18)

    def record(site, layer, exact, rounded):
        v = probe(site, layer, exact, rounded)
        stored[(site, layer)] = v.copy()
        return v

    other, _ = forward_block(shape, w, [], toks, depth, vis, rounding=record)
    chk = RoundingCheck(stored)
    got, _ = forward_block(shape, w, [], toks, depth, vis, rounding=chk)
    assert chk.mismatches() == 0 and chk.flips() > 0, chk.summary()
    np.testing.assert_allclose(got, other, rtol=0, atol=1e-12)

    bad = dict(stored)
    z = bad[("z", 1)].copy()
    z.flat[5] = round_bf16(z.flat[5] * (1 + 2 * 2.0 ** -7))
    bad[("z", 1)] = z
    chk = RoundingCheck(bad)
    forward_block(shape, w, [], toks, depth, vis, rounding=chk)
    assert chk.mismatches() == 1, chk.summary()
