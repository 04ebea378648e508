"""Pins of the oracle's per-operation arithmetic against closed forms,
identities and library routines (CPU only)."""

import numpy as np
import pytest
import torch
from scipy.special import expit

from oracle.model import attention, rmsnorm, rope, silu
from oracle.numerics import round_bf16


def _torch_bf16(x32):
    return torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()


def test_round_bf16_matches_torch_casts():
    g = np.random.default_rng(0)
    x = (g.standard_normal(200000) * np.exp(g.uniform(-30, 30, 200000))).astype(np.float32)
    np.testing.assert_array_equal(round_bf16(x.astype(np.float64)), _torch_bf16(x))


def test_round_bf16_ties_subnormals_overflow():
    bits = []
    for hi in (0x3F80, 0x3F81, 0xBF80, 0xBF81, 0x0001, 0x0002, 0x0080, 0x8001, 0x7F7F, 0xFF7F):
        for lo in (0x0000, 0x7FFF, 0x8000, 0x8001, 0xFFFF):
            bits.append((hi << 16) | lo)
    x = np.array(bits, dtype=np.uint32).view(np.float32)
    x = x[np.isfinite(x)]
    got = round_bf16(x.astype(np.float64))
    np.testing.assert_array_equal(got, _torch_bf16(x))
    # exact halfway between 1 and the next bf16 value rounds to the even one (1.0)
    assert round_bf16(1.0 + 2.0 ** -8) == 1.0
    assert round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6
    assert np.isinf(round_bf16(3.5e38))


def test_rope_position_zero_is_identity_and_preserves_norm():
    g = np.random.default_rng(1)
    u = g.standard_normal((5, 3, 64))
    np.testing.assert_array_equal(rope(u, np.zeros(5), 10000.0), u)
    r = rope(u, np.arange(5) * 37, 10000.0)
    np.testing.assert_allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(u, axis=-1), rtol=1e-12)


def test_rope_dot_product_depends_only_on_offset():
    g = np.random.default_rng(2)
    q = g.standard_normal((1, 1, 128))
    k = g.standard_normal((1, 1, 128))
    dots = []
    for m in (5, 100, 2043):
        rq = rope(q, np.array([m + 7]), 10000.0)
        rk = rope(k, np.array([m]), 10000.0)
        dots.append(float(np.sum(rq * rk)))
    np.testing.assert_allclose(dots, dots[0], rtol=1e-10)


def test_rope_matches_complex_rotation():
    """Pair (u_i, u_{i+hd/2}) as the complex number u_i + i u_{i+hd/2}; RoPE
    multiplies it by exp(i * pos * theta^(-2i/hd))."""
    g = np.random.default_rng(3)
    hd = 16
    u = g.standard_normal((4, 2, hd))
    pos = np.array([0, 1, 9, 300])
    z = u[..., : hd // 2] + 1j * u[..., hd // 2:]
    w = np.exp(1j * pos[:, None, None] * 10000.0 ** (-np.arange(hd // 2) * 2.0 / hd))
    zr = z * w
    ref = np.concatenate([zr.real, zr.imag], axis=-1)
    np.testing.assert_allclose(rope(u, pos, 10000.0), ref, rtol=1e-12, atol=1e-12)


def test_rmsnorm_output_has_unit_rms_and_matches_torch():
    g = np.random.default_rng(4)
    h = g.standard_normal((6, 256)) * 3.0
    x = rmsnorm(h, np.ones(256), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(x * x, axis=-1)), 1.0, rtol=1e-12)
    gain = 1.0 + 0.1 * g.standard_normal(256)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(h), (256,), torch.from_numpy(gain), eps=1e-5)
    np.testing.assert_allclose(rmsnorm(h, gain, 1e-5), ref.numpy(), rtol=1e-12)


def test_silu_closed_form():
    t = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(silu(t), t * expit(t), rtol=1e-12, atol=1e-300)
    assert silu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(silu(torch.linspace(-5, 5, 11, dtype=torch.float64).numpy()),
                               torch.nn.functional.silu(torch.linspace(-5, 5, 11, dtype=torch.float64)).numpy(),
                               rtol=1e-12)


def test_attention_single_visible_key_returns_its_value():
    g = np.random.default_rng(5)
    q = g.standard_normal((3, 4, 8))
    keys = g.standard_normal((5, 2, 8))
    vals = g.standard_normal((5, 2, 8))
    mask = np.zeros((3, 5), dtype=bool)
    mask[0, 2] = mask[1, 0] = mask[2, 4] = True
    o = attention(q, keys, vals, mask, 0.3)
    for r, c in ((0, 2), (1, 0), (2, 4)):
        for j in range(4):
            np.testing.assert_array_equal(o[r, j], vals[c, j // 2])


def test_attention_equal_scores_average_values_and_matches_sdpa():
    g = np.random.default_rng(6)
    vals = g.standard_normal((7, 1, 4))
    q = np.zeros((1, 1, 4))
    keys = g.standard_normal((7, 1, 4))
    o = attention(q, keys, vals, np.ones((1, 7), dtype=bool), 1.0)
    np.testing.assert_allclose(o[0, 0], vals[:, 0].mean(axis=0), rtol=1e-12)
    # against torch's scaled_dot_product_attention with a causal mask (MHA)
    T, H, hd = 6, 3, 16
    q = g.standard_normal((T, H, hd))
    k = g.standard_normal((T, H, hd))
    v = g.standard_normal((T, H, hd))
    mask = np.tril(np.ones((T, T), dtype=bool))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).transpose(0, 1), torch.from_numpy(k).transpose(0, 1),
        torch.from_numpy(v).transpose(0, 1), is_causal=True).transpose(0, 1).numpy()
    np.testing.assert_allclose(attention(q, k, v, mask, 1 / np.sqrt(hd)), ref, rtol=1e-10, atol=1e-12)


def test_gqa_groups_are_contiguous():
    """With 4 query heads over 2 KV heads, heads 0,1 read KV head 0 and heads
    2,3 read KV head 1: identical to MHA with each KV head duplicated."""
    g = np.random.default_rng(7)
    q = g.standard_normal((5, 4, 8))
    k = g.standard_normal((9, 2, 8))
    v = g.standard_normal((9, 2, 8))
    mask = np.ones((5, 9), dtype=bool)
    mha = attention(q, np.repeat(k, 2, axis=1), np.repeat(v, 2, axis=1), mask, 0.5)
    np.testing.assert_allclose(attention(q, k, v, mask, 0.5), mha, rtol=1e-13)


def test_norm_scale_times_gained_input_is_rmsnorm():
    """The split form used before a projection: r * (h * g) with r the row's
    RMS scale equals RMSNorm(h) * g, with r from torch's rms_norm of a ones
    gain as an independent reference."""
    from oracle.model import norm_scale
    g = np.random.default_rng(4)
    h = g.standard_normal((5, 192)) * 3.0
    gain = 1.0 + 0.1 * g.standard_normal(192)
    np.testing.assert_allclose(norm_scale(h, 1e-5) * (h * gain), rmsnorm(h, gain, 1e-5), rtol=1e-13)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(h), (192,), torch.ones(192, dtype=torch.float64), 1e-5)
    np.testing.assert_allclose(norm_scale(h, 1e-5) * h, ref.numpy(), rtol=1e-12)
