"""GPU parity of the verification step against the CPU oracle, through the C ABI."""

import numpy as np
import pytest

from oracle import OracleSession
from oracle.numerics import to_f64
from tests.helpers import assert_step_matches, reuse_session_parity
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


def test_tiny_fp32_reuse_session_matches_oracle(ee):
    """64-token prompt of a 192-token Zipf 'original code', then 16 Reuse
    verify steps of K = 8 with drafts at the matcher's offset."""
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=1234)
    code = zipf_tokens(shape.vocab, 192, seed=42)
    eng = ee.Engine(shape, w, max_ctx=256, k_max=8)
    ref, compared, unpinned = reuse_session_parity(eng, shape, w, code[:64], code, steps=16, k=8, tol=1e-4)
    assert compared == 16 and unpinned == 0
    for l in range(shape.n_layers):
        k, v = eng.read_kv(0, l)
        np.testing.assert_allclose(k, ref.cache[l][0], rtol=0, atol=2e-5)
        np.testing.assert_allclose(v, ref.cache[l][1], rtol=0, atol=2e-5)
    eng.close()


@pytest.mark.parametrize("std", [0.1])
def test_tiny_fp32_planted_drafts_accept_exactly(ee, std):
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=77, std=std)
    prompt = zipf_tokens(shape.vocab, 40, seed=5)
    ref = OracleSession(shape, w)
    ref.prefill(prompt)
    eng = ee.Engine(shape, w, max_ctx=256, k_max=16)
    eng.prefill(0, prompt)
    g = np.random.default_rng(0)
    for step in range(12):
        probe = OracleSession(shape, w)
        probe.set_cache(ref.cache, ref.pending)
        truth = probe.greedy(17)
        k = int(g.integers(0, 17))
        j = int(g.integers(0, k + 1))
        d = planted_draft(truth, j, k, shape.vocab, seed=step)
        ra, rn, _ = ref.verify(d)
        a, n, _ = eng.verify(0, d)
        assert_step_matches(eng.logits(), a, n, ref.last_logits, ra, rn, k, 1e-4)
        assert ra == j
    eng.close()


def test_bf16_gqa_session_matches_oracle(ee):
    """Six Reuse steps of K = 32 (GQA, random gains); every step compared,
    near ties decided the GPU's way followed by the oracle (G12)."""
    shape = _bf16_small()
    w = gen_weights(shape, seed=21, gains="random")
    code = zipf_tokens(shape.vocab, 400, seed=8)
    eng = ee.Engine(shape, w, max_ctx=512, k_max=32)
    ref, compared, unpinned = reuse_session_parity(eng, shape, w, code[:150], code, steps=6, k=32, tol=2e-2)
    print(f"bf16 session: {compared} steps compared, {unpinned} near ties followed")
    assert compared == 6 and unpinned <= 2
    for l in range(shape.n_layers):
        k, v = eng.read_kv(0, l)
        rk, rv = ref.cache[l]
        assert len(k) == len(rk)
        for got, want in ((k, rk), (v, rv)):
            assert np.abs(to_f64(got, "bf16") - want).max() <= 2e-2 * max(1.0, np.abs(want).max())
    eng.close()


def test_bf16_prefill_longer_than_block_matches_oracle(ee):
    """Prefill in several blocks across page and split boundaries."""
    shape = _bf16_small(n_layers=1)
    w = gen_weights(shape, seed=3)
    prompt = zipf_tokens(shape.vocab, 300, seed=9)
    ref = OracleSession(shape, w)
    p = ref.prefill(prompt)
    eng = ee.Engine(shape, w, max_ctx=512, k_max=16)
    q = eng.prefill(0, prompt)
    lg = eng.logits()
    np.testing.assert_allclose(lg, ref.last_logits[-len(lg):], rtol=0, atol=2e-2)
    assert p == q or float(np.sort(ref.last_logits[-1])[-1] - np.sort(ref.last_logits[-1])[-2]) <= 2e-2
    eng.close()


def test_bf16_width_not_a_multiple_of_256_matches_oracle(ee):
    """d = 1280: 40 super-steps of 32 columns, not a multiple of the 8 waves
    that split a projection's reduction, so part of every wave's register and
    LDS fragments lie past K.  Drafts of 64 tokens make 65-row blocks (two row
    groups, the second with a 33rd row held in LDS); GQA with 5 query heads per
    KV head."""
    shape = _bf16_small(n_layers=1, d_model=1280, n_heads=10, n_kv_heads=2, ffn=2560)
    w = gen_weights(shape, seed=31, gains="random")
    code = zipf_tokens(shape.vocab, 400, seed=12)
    eng = ee.Engine(shape, w, max_ctx=512, k_max=64)
    ref, compared, unpinned = reuse_session_parity(eng, shape, w, code[:150], code, steps=3, k=64, tol=2e-2)
    assert compared == 3 and unpinned <= 1
    k, v = eng.read_kv(0, 0)
    rk, rv = ref.cache[0]
    assert len(k) == len(rk)
    for got, want in ((k, rk), (v, rv)):
        assert np.abs(to_f64(got, "bf16") - want).max() <= 2e-2 * max(1.0, np.abs(want).max())
    eng.close()
