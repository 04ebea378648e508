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
