"""Error handling and state rules of the C ABI on the GPU."""

import numpy as np
import pytest

from workloads import gen_weights, get_shape, zipf_tokens

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ee():
    import paper_2506_02780_amd as mod
    return mod


@pytest.fixture(scope="module")
def eng(ee):
    shape = get_shape("tiny")
    e = ee.Engine(shape, gen_weights(shape, seed=9, std=0.1), max_ctx=200, max_seqs=2, k_max=8)
    yield e
    e.close()


def _expect(ee, code, fn, *args):
    with pytest.raises(ee.EEError) as ex:
        fn(*args)
    assert ex.value.code == code


def test_verify_before_prefill_and_bad_arguments(ee, eng):
    _expect(ee, ee.EE_ESTATE, eng.verify, 1, [1, 2])
    p = eng.prefill(1, zipf_tokens(1024, 20, seed=1))
    state = eng.seq_state(1)
    _expect(ee, ee.EE_EINVAL, eng.verify, 1, list(range(9)))           # K > k_max
    _expect(ee, ee.EE_EINVAL, eng.verify, 1, [1, 5000])                 # token >= vocab
    _expect(ee, ee.EE_EINVAL, eng.verify, 1, [1, 2, 3], [0, -1, 1])     # parent[0] must be -1
    _expect(ee, ee.EE_EINVAL, eng.verify, 1, [1, 2, 3], [-1, 1, 0])     # parent[1] >= 1
    _expect(ee, ee.EE_ESTATE, eng.rollback, 1, 21, 3)                   # beyond the length
    _expect(ee, ee.EE_EINVAL, eng.verify, 5, [1])                       # no such sequence
    _expect(ee, ee.EE_ESTATE, eng.prefill, 1, [1, 2])                   # already live
    assert eng.seq_state(1) == state == (20, p)
    eng.rollback(1, 0, -1)
    assert eng.seq_state(1) == (0, -1)


def test_capacity_errors_leave_state_unchanged(ee, eng):
    p = eng.prefill(0, zipf_tokens(1024, 195, seed=2))
    _expect(ee, ee.EE_ECAPACITY, eng.verify, 0, list(range(8)))         # 195 + 9 rows > max_ctx 200
    assert eng.seq_state(0) == (195, p)
    a, nxt, _ = eng.verify(0, [1, 2])
    assert eng.seq_state(0) == (196 + a, nxt)
    _expect(ee, ee.EE_ECAPACITY, eng.prefill, 1, zipf_tokens(1024, 250, seed=3))
    assert eng.seq_state(1) == (0, -1)
    # a length at the top of the int32 range is refused before any token is read
    import ctypes
    buf = (ctypes.c_int32 * 4)(1, 2, 3, 4)
    nx = ctypes.c_int32()
    assert ee.ee_prefill(eng.ctx, 1, buf, 2 ** 31 - 1, ctypes.byref(nx)) == ee.EE_ECAPACITY
    assert eng.seq_state(1) == (0, -1)
    eng.rollback(0, 0, -1)


def test_rollback_then_regenerate_is_bitwise_identical(ee, eng):
    prompt = zipf_tokens(1024, 33, seed=4)
    first = eng.prefill(0, prompt)
    s1 = [eng.verify(0, [])[1] for _ in range(10)]
    lg1 = eng.logits()
    eng.rollback(0, 33, first)
    s2 = [eng.verify(0, [])[1] for _ in range(10)]
    assert s1 == s2
    np.testing.assert_array_equal(eng.logits(), lg1)
    eng.rollback(0, 0, -1)


def test_time_gemm_measurement_aid(ee, eng):
    us = eng.time_gemm("gateup", 9, reps=2)
    assert 0.0 < us < 1e5
    n0 = eng.seq_state(0)
    for bad in (("attn", 9), ("gateup", 0), ("gateup", 10 ** 6)):
        with pytest.raises(ee.EEError) as e:
            eng.time_gemm(*bad)
        assert e.value.code == ee.EE_EINVAL
    assert eng.seq_state(0) == n0


def test_time_stream_read_measurement_aid(ee, eng):
    import torch
    buf = torch.empty((1 << 20) + 48, dtype=torch.uint8, device="cuda")   # a partial last segment
    us = eng.time_stream_read(buf, reps=2)
    assert 0.0 < us < 1e5
    with pytest.raises(ee.EEError) as e:
        eng.time_stream_read(buf[:1 << 17], reps=1)   # below 256 KiB
    assert e.value.code == ee.EE_EINVAL


def test_load_kv_round_trip_errors_and_parity(ee, eng):
    """ee_load_kv installs a cache that ee_read_kv returns unchanged; a block
    over it matches the oracle over the same cache (fp32, 1e-4); errors leave
    the sequence empty."""
    from oracle import OracleSession
    from workloads import random_kv_context
    shape = get_shape("tiny")
    n = 150   # three pages, the last one partly filled
    kv = random_kv_context(shape.n_layers, n, shape.n_kv_heads, shape.head_dim, seed=8, dtype="f32")
    k = np.stack([a for a, _ in kv])
    v = np.stack([b for _, b in kv])
    _expect(ee, ee.EE_EINVAL, eng.load_kv, 1, k, v, shape.vocab)       # pending outside [0, vocab)
    _expect(ee, ee.EE_ECAPACITY, eng.load_kv, 1,
            np.zeros((shape.n_layers, 200, shape.n_kv_heads, shape.head_dim), np.float32),
            np.zeros((shape.n_layers, 200, shape.n_kv_heads, shape.head_dim), np.float32), 3)   # n + 1 > max_ctx
    assert eng.seq_state(1) == (0, -1)
    eng.load_kv(1, k, v, 17)
    assert eng.seq_state(1) == (n, 17)
    _expect(ee, ee.EE_ESTATE, eng.load_kv, 1, k, v, 17)                 # not empty
    for l in range(shape.n_layers):
        rk, rv = eng.read_kv(1, l)
        np.testing.assert_array_equal(rk, k[l])
        np.testing.assert_array_equal(rv, v[l])
    w = gen_weights(shape, seed=9, std=0.1)   # the engine's weights
    ref = OracleSession(shape, w)
    ref.set_cache([(a.astype(np.float64), b.astype(np.float64)) for a, b in kv], 17)
    d = zipf_tokens(shape.vocab, 8, seed=6)
    ra, rn, _ = ref.verify(d)
    a, nxt, _ = eng.verify(1, d)
    np.testing.assert_allclose(eng.logits(), ref.last_logits, rtol=0, atol=1e-4)
    assert (a, nxt) == (ra, rn)
    eng.rollback(1, 0, -1)
