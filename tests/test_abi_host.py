"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function the header declares, sizes configs, rejects bad configs before
touching the GPU, and its matcher equals the oracle's."""

import ctypes
import os
import re

import numpy as np
import pytest

from workloads import get_shape

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2506_02780_amd", "libee.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libee.so not built")


def _declared():
    src = open(os.path.join(ROOT, "include", "ee.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ee_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    import paper_2506_02780_amd as ee
    names = _declared()
    assert len(names) >= 12
    for n in names:
        assert hasattr(ee._lib, n), n


def test_config_sizes_and_validation():
    import paper_2506_02780_amd as ee
    cfg = ee.make_config(get_shape("7b"), max_ctx=2048 + 65, k_max=64)
    p = ctypes.byref(cfg)
    packed = ee.ee_packed_weight_bytes(p)
    # every linear weight plus embedding, gains and alignment padding
    assert 2 * 5.9e9 < packed < 2 * 6.0e9
    assert ee.ee_kv_pool_bytes(p) == 32 * 34 * 2 * 8 * 64 * 128 * 2   # 34 pages of 64 positions
    assert ee.ee_workspace_bytes(p) > 0
    bad = ee.make_config(get_shape("7b", head_dim=96), max_ctx=128)
    assert ee.ee_workspace_bytes(ctypes.byref(bad)) == 0
    ctx = ctypes.c_void_p()
    w = ee.EEWeights()
    rc = ee.ee_create(ctypes.byref(bad), ctypes.byref(w), 1, 1, 1, None, ctypes.byref(ctx))
    assert rc == ee.EE_EINVAL and b"head_dim" in ee.ee_last_error(None)
    assert ee.ee_destroy(None) == ee.EE_EINVAL
    # an LM head of 2 GiB or more (vocab 152064 x d 8192 in bf16) is refused:
    # it is addressed with 32-bit offsets
    huge = ee.make_config(get_shape("7b", d_model=8192, vocab=152064), max_ctx=128)
    assert ee.ee_workspace_bytes(ctypes.byref(huge)) == 0
    rc = ee.ee_create(ctypes.byref(huge), ctypes.byref(w), 1, 1, 1, None, ctypes.byref(ctx))
    assert rc == ee.EE_EINVAL and b"LM head" in ee.ee_last_error(None)
    assert ee.ee_capture_bytes(ctypes.byref(cfg), 33) > 0 and ee.ee_capture_bytes(ctypes.byref(cfg), 0) == 0
    # n_heads * head_dim beyond the int range (2^25 x 128 = 2^32) is refused, not wrapped
    wide = ee.make_config(get_shape("7b", n_heads=2 ** 25, n_kv_heads=2 ** 25), max_ctx=128)
    assert ee.ee_workspace_bytes(ctypes.byref(wide)) == 0
    rc = ee.ee_create(ctypes.byref(wide), ctypes.byref(w), 1, 1, 1, None, ctypes.byref(ctx))
    assert rc == ee.EE_EINVAL and b"n_heads*head_dim" in ee.ee_last_error(None)


def test_null_context_calls_fail_cleanly():
    import paper_2506_02780_amd as ee
    a = ctypes.c_int32()
    assert ee.ee_verify(None, 0, None, 0, None, ctypes.byref(a), ctypes.byref(a), None) == ee.EE_EINVAL
    assert ee.ee_kv_rollback(None, 0, 0, 0) == ee.EE_EINVAL
    assert ee.ee_verify_batch(None, 1, None, None, 0, None, None, None, None) == ee.EE_EINVAL
    assert ee.ee_verify_topk(None, 1, None, None, 0, 3, 1, None, None, None) == ee.EE_EINVAL
    assert ee.ee_extend(None, 0, None, 0, ctypes.byref(a)) == ee.EE_EINVAL
    assert ee.ee_time_gemm(None, 5, 1, 1, None) == ee.EE_EINVAL
    assert ee.ee_time_stream_read(None, None, 16, 1, None) == ee.EE_EINVAL
    assert ee.ee_capture(None, None, 0) == ee.EE_EINVAL
    assert ee.ee_verify_noalloc(None, 0, None, 0, None, ctypes.byref(a), ctypes.byref(a), None) == ee.EE_EINVAL
    assert ee.ee_edit_begin(None, 0, None, 0, None) == ee.EE_EINVAL


def test_matcher_equals_oracle():
    import paper_2506_02780_amd as ee
    from oracle import match_reuse
    g = np.random.default_rng(3)
    for _ in range(2000):
        orig = g.integers(0, 4, int(g.integers(0, 30)))
        gen = g.integers(0, 4, int(g.integers(0, 12)))
        cur = int(g.integers(0, len(orig) + 3))
        lo = int(g.integers(1, 3))
        hi = int(g.integers(lo, 9))
        assert ee.match_reuse(gen, orig, cur, lo, hi) == match_reuse(gen, orig, cur, lo, hi)
    # cursors at the ends of the int32 range (no bound / nothing left to draft)
    for _ in range(200):
        orig = g.integers(0, 3, int(g.integers(0, 30)))
        gen = g.integers(0, 3, int(g.integers(1, 8)))
        for cur in (-2 ** 31, -2 ** 31 + 1, -7, 2 ** 31 - 1):
            assert ee.match_reuse(gen, orig, cur, 1, 4) == match_reuse(gen, orig, cur, 1, 4)
    a = ctypes.c_int32()
    assert ee.ee_match_reuse_c(None, 0, None, 0, 0, 0, 8, ctypes.byref(a), ctypes.byref(a)) == ee.EE_EINVAL
