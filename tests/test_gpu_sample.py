"""Stochastic speculative verification (ee_verify_sample, Eq. 4) through the
C ABI, against the oracle on its own logits.  A decision is compared where
it is unique: the acceptance test eps q < p is further from equality than
the logit error can move it, and the resampling target lies further from
every cumulative-weight boundary."""

import numpy as np
import pytest

from oracle import OracleSession, accept_sample, target_probs
from workloads import gen_weights, get_shape, planted_draft, zipf_tokens

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ee():
    import paper_2506_02780_amd as mod
    return mod


def _unique(draft, logits, eps, u, q, temp, residual, err):
    """True when a perturbation of every logit by err cannot change the
    oracle's decisions (first-order bound on p: |dp| <= 2 p err / temp)."""
    K = len(draft)
    for i in range(K + 1):
        p = target_probs(logits[i], temp)
        dp = 2 * p * err / temp + 1e-12
        if i < K:
            d = draft[i]
            qd = 1.0 if q is None else float(q[i][d])
            if abs(eps[i] * qd - p[d]) <= dp[d]:
                return False
            if eps[i] * qd < p[d]:
                continue
            if residual:
                qi = np.zeros_like(p)
                if q is None:
                    qi[d] = 1.0
                else:
                    qi = np.asarray(q[i], dtype=np.float64)
                w = np.maximum(p - qi, 0)        # moves by at most dp per token, as p does
                dw = dp
            else:
                w, dw = p, dp
        else:
            w, dw = p, dp
        c = np.cumsum(w)
        tgt = u[i] * c[-1]
        slack = np.cumsum(dw)[-1] * 2
        return bool(np.min(np.abs(c - tgt)) > slack)
    return True


@pytest.mark.parametrize("draft_kind,residual,temp", [("q", True, 1.0), ("q", False, 1.0), ("greedy", True, 0.7),
                                                       ("greedy", False, 1.3)])
def test_sample_verification_matches_oracle(ee, draft_kind, residual, temp):
    """Trials from one committed state (the GPU is rolled back after each):
    planted drafts, random draft distributions (or a greedy draft) and draws."""
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=31, std=0.1)
    w.final_gain = (w.final_gain * 3.0).astype(np.float32)     # rows with some dominant tokens
    prompt = zipf_tokens(shape.vocab, 50, seed=32)
    ref = OracleSession(shape, w)
    ref.prefill(prompt)
    truth = OracleSession(shape, w)
    truth.set_cache(ref.cache, ref.pending)
    cont = truth.greedy(9)
    eng = ee.Engine(shape, w, max_ctx=512, k_max=16)
    eng.prefill(0, prompt)
    n0, p0 = eng.seq_state(0)
    g = np.random.default_rng(33 + residual)
    compared = 0
    outcomes = set()
    for trial in range(40):
        K = int(g.integers(0, 9))
        draft = planted_draft(cont, int(g.integers(0, K + 1)), K, shape.vocab, seed=trial)
        q = None
        if draft_kind == "q":
            q = g.dirichlet(np.full(shape.vocab, 0.05), size=K).astype(np.float32)
            for i, d in enumerate(draft):
                q[i, d] += 0.5                       # the drafted token is likely under q
            q /= q.sum(axis=1, keepdims=True)
        eps = g.random(K).astype(np.float32)
        u = g.random(K + 1).astype(np.float32)
        ga, gn = eng.verify_sample(0, draft, eps, u, q, temp, residual)
        assert eng.seq_state(0) == (n0 + 1 + ga, gn)
        gl = eng.logits()
        eng.rollback(0, n0, p0)
        rl = ref.score(draft)
        err = float(np.abs(gl - rl).max())
        assert err <= 3 * 1e-4           # the stated fp32 tolerance, scaled with the logits (gain x3)
        e64, u64 = eps.astype(np.float64), u.astype(np.float64)
        ra, rn = accept_sample(draft, rl, e64, u64, q, temp, residual)
        if _unique(list(draft), rl, e64, u64, q, temp, residual, err):
            assert (ga, gn) == (ra, rn), (trial, ga, gn, ra, rn)
            compared += 1
            outcomes.add((ga == K, ga))
    eng.close()
    assert compared >= 25
    assert len(outcomes) >= 3                        # rejections at several rows and full acceptance


def test_greedy_draft_at_low_temperature_is_greedy_verification(ee):
    shape = get_shape("tiny")
    w = gen_weights(shape, seed=34, std=0.1)
    prompt = zipf_tokens(shape.vocab, 40, seed=35)
    eng = ee.Engine(shape, w, max_ctx=512, k_max=16)
    eng.prefill(0, prompt)
    n0, p0 = eng.seq_state(0)
    cont = [eng.verify(0, [])[1] for _ in range(12)]
    eng.rollback(0, n0, p0)
    g = np.random.default_rng(36)
    for trial in range(10):
        K = int(g.integers(1, 11))
        d = planted_draft(cont, int(g.integers(0, K + 1)), K, shape.vocab, seed=trial)
        a, nxt, _ = eng.verify(0, d)
        eng.rollback(0, n0, p0)
        sa, sn = eng.verify_sample(0, d, g.random(K) * 0.99, g.random(K + 1) * 0.99, None, 1e-4, True)
        eng.rollback(0, n0, p0)
        assert (sa, sn) == (a, nxt)
    with pytest.raises(ee.EEError) as e:
        eng.verify_sample(0, [1, 2], [0.5, 1.0], [0.1, 0.2, 0.3])
    assert e.value.code == ee.EE_EINVAL
    with pytest.raises(ee.EEError) as e:
        eng.verify_sample(0, [1, 2], [0.5, 0.5], [0.1, 0.2, 0.3], temperature=0.0)
    assert e.value.code == ee.EE_EINVAL
    assert eng.seq_state(0) == (n0, p0)
    eng.close()
