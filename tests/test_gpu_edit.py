"""Edit sessions (ee_edit_begin / ee_edit_step): the Reuse / Generate phase
machine with an optional draft model, through the C ABI, against the
oracle's driver."""

import numpy as np
import pytest

from oracle import OracleEditSession, OracleSession
from workloads import gen_weights, get_shape, inject_edits, zipf_tokens

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ee():
    import paper_2506_02780_amd as mod
    return mod


def _workload(shape, w, n_prompt, n_out, seed, frac):
    prompt = zipf_tokens(shape.vocab, n_prompt, seed=seed)
    ref = OracleSession(shape, w)
    ref.prefill(prompt)
    greedy = [ref.pending] + ref.greedy(n_out - 1)
    original, _ = inject_edits(np.asarray(greedy, dtype=np.int32), shape.vocab, seed=seed + 1, frac=frac)
    return prompt, greedy, original


@pytest.mark.parametrize("draft_kind,top_k", [(None, 0), ("same", 0), ("other", 0), ("other", 5), ("same", 3)])
def test_edit_session_matches_oracle_driver(ee, draft_kind, top_k):
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=5, std=0.1)
    prompt, greedy, original = _workload(shape, w, 40, 120, seed=6, frac=0.15)
    dshape, dw = shape, w
    if draft_kind == "other":
        dshape = get_shape("tiny", n_layers=1)
        dw = gen_weights(dshape, seed=105, std=0.1)
    # oracle
    t_ref = OracleSession(shape, w)
    t_ref.prefill(prompt)
    d_ref = None
    if draft_kind:
        d_ref = OracleSession(dshape, dw)
        d_ref.prefill(prompt)
    ref = OracleEditSession(t_ref, original, d_ref, k_reuse=8, gamma=4, top_k=top_k, dynamic=True, min_match=3)
    # GPU
    tgt = ee.Engine(shape, w, max_ctx=512, k_max=16)
    tgt.prefill(0, prompt)
    drf = None
    if draft_kind:
        drf = ee.Engine(dshape, dw, max_ctx=512, k_max=16)
        drf.prefill(0, prompt)
    s = ee.EditSession(tgt, 0, original, drf, 0, k_reuse=8, gamma=4, top_k=top_k, dynamic=True, min_match=3)
    phases = set()
    while len(ref.out) < 120:
        rp, rnew = ref.step()
        gp, gnew = s.step()
        assert (gp, gnew) == (rp, rnew), (len(ref.out), gp, gnew, rp, rnew)
        phases.add(gp)
        assert s.state.phase == ref.phase and s.state.cursor == ref.cursor
        assert tgt.seq_state(0) == (t_ref.n, t_ref.pending)
        if drf is not None:
            assert drf.seq_state(0) == (d_ref.n, d_ref.pending)
    assert s.output == ref.out
    assert phases == {ee.EE_PHASE_REUSE, ee.EE_PHASE_GENERATE}
    if top_k == 0:
        assert s.output[:len(greedy)] == greedy
    if draft_kind:
        assert s.state.draft_tokens > 0 and s.state.steps[1] > 0
    tgt.close()
    if drf is not None:
        drf.close()


def test_edit_session_with_greedy_verification_is_lossless_bitwise(ee):
    """bf16 target, a different 1-layer bf16 draft model: with Eq. 7 in both
    phases the session output equals the GPU's own greedy decoding."""
    shape = get_shape("tiny", n_layers=2, d_model=512, n_heads=4, n_kv_heads=2, head_dim=128, ffn=1024,
                      vocab=2048, dtype="bf16")
    w = gen_weights(shape, seed=61, std=0.05)
    dshape = get_shape("tiny", n_layers=1, d_model=512, n_heads=4, n_kv_heads=2, head_dim=128, ffn=1024,
                       vocab=2048, dtype="bf16")
    dw = gen_weights(dshape, seed=62, std=0.05)
    prompt = zipf_tokens(shape.vocab, 150, seed=63)
    tgt = ee.Engine(shape, w, max_ctx=1024, k_max=32)
    first = tgt.prefill(0, prompt)
    greedy = [first] + [tgt.verify(0, [])[1] for _ in range(299)]
    tgt.rollback(0, len(prompt), first)
    original, _ = inject_edits(np.asarray(greedy, dtype=np.int32), shape.vocab, seed=64, frac=0.1)
    drf = ee.Engine(dshape, dw, max_ctx=1024, k_max=32)
    drf.prefill(0, prompt)
    s = ee.EditSession(tgt, 0, original, drf, 0, k_reuse=32, gamma=7, top_k=0)
    while s.n < 300:
        s.step()
    assert s.output[:300] == greedy
    st = s.state
    assert st.steps[0] > 0 and st.steps[1] > 0 and st.emitted[0] > st.emitted[1]
    tgt.close()
    drf.close()


def test_edit_session_errors(ee):
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=3)
    tgt = ee.Engine(shape, w, max_ctx=256, k_max=8)
    drf = ee.Engine(shape, w, max_ctx=256, k_max=8)
    tgt.prefill(0, zipf_tokens(shape.vocab, 30, seed=1))
    drf.prefill(0, zipf_tokens(shape.vocab, 31, seed=1))
    with pytest.raises(ee.EEError) as e:          # the draft holds a different prompt length
        ee.EditSession(tgt, 0, list(range(50)), drf, 0)
    assert e.value.code == ee.EE_ESTATE
    s = ee.EditSession(tgt, 0, list(range(50)), None, 0, k_reuse=8)
    before = tgt.seq_state(0)
    s._out[0] = (before[1] + 1) % shape.vocab     # output that does not end with the pending token
    with pytest.raises(ee.EEError) as e:
        s.step()
    assert e.value.code == ee.EE_ESTATE
    s._out[0] = before[1]
    s.params.k_reuse = 0
    with pytest.raises(ee.EEError) as e:
        s.step()
    assert e.value.code == ee.EE_EINVAL
    s.params.k_reuse = 9                           # beyond k_max: the verify call refuses it
    with pytest.raises(ee.EEError) as e:
        s.step()
    assert e.value.code == ee.EE_EINVAL
    assert tgt.seq_state(0) == before
    s.params.k_reuse = 8
    s.state.cursor = -1                            # the fallback draft would start before the original
    with pytest.raises(ee.EEError) as e:
        s.step()
    assert e.value.code == ee.EE_EINVAL
    assert tgt.seq_state(0) == before
    s.state.cursor = 0
    s.step()
    assert tgt.seq_state(0)[0] > before[0]
    tgt.close()
    drf.close()
