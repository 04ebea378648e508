"""Oracle forward of the target model over one block of rows (test infrastructure only).

Eq. 3 scores a draft appended to the already-processed prefix in one forward
of the target model.  Here the prefix is represented by its committed key /
value cache (n positions) and the block holds T rows.  Row r sits at position
n + depth[r] and sees every committed key plus the block rows that are its
ancestors or itself (a chain for a linear draft, the root-to-node path for a
draft tree).

The decoder is the usual Llama-style stack (the paper's targets are
decoder-only code LLMs; its text does not spell the layers out):

    h   = E[token]
    per layer:
      x = RMSNorm(h) * g_attn                 x = h / sqrt(mean(h^2) + eps)
      q, k, v = x Wq^T, x Wk^T, x Wv^T        split into heads of size hd
      q, k = RoPE(q, pos), RoPE(k, pos)       rotate-half pairs (i, i + hd/2),
                                              angle pos * theta^(-2i/hd)
      query head j reads key/value head floor(j * Hkv / H)
      o = softmax(q k^T / sqrt(hd)) v         over the visible keys
      h = h + o Wo^T
      x = RMSNorm(h) * g_ffn
      h = h + (silu(x Wg^T) * (x Wu^T)) Wd^T  silu(t) = t / (1 + e^-t)
    logits = (RMSNorm(h) * g_final) Wlm^T

Everything is float64.  For bf16 models, the quantities a bf16 pipeline
stores in bf16 are rounded to bf16 (nearest-even): the inputs of the
projections that follow a norm, q and k after RoPE, v (so the cache holds
bf16 keys and values), the attention output o and the SwiGLU product.
Residual stream, scores, softmax and logits stay float64.  fp32 models are
not rounded at all.

A norm followed by a projection, RMSNorm(h) * g W^T, is evaluated as
r * ((h * g) W^T) with the row's scale r = 1 / sqrt(mean(h^2) + eps): the
same value, with h * g as the quantity that is stored (and so rounded) before
the projection.
"""

from __future__ import annotations

import numpy as np

from .numerics import round_bf16, to_f64


def _rounder(dtype: str):
    return round_bf16 if dtype == "bf16" else (lambda a: a)


def rmsnorm(h, gain, eps):
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps) * gain


def norm_scale(h, eps):
    """The RMSNorm scale of every row of h: 1 / sqrt(mean(h^2) + eps), shape [T, 1]."""
    return 1.0 / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps)


def rope(u, pos, theta):
    """u: [T, heads, hd]; pos: [T].  Rotate-half pairing."""
    hd = u.shape[-1]
    half = hd // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    a, b = u[..., :half], u[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(t):
    return t / (1.0 + np.exp(-t))


def attention(q, keys, vals, mask, scale):
    """q: [T, H, hd]; keys, vals: [S, Hkv, hd]; mask: [T, S] visibility.
    Query head j reads key/value head floor(j * Hkv / H).  Returns [T, H, hd]."""
    t, H, hd = q.shape
    Hkv = keys.shape[1]
    o = np.empty((t, H, hd))
    for j in range(H):
        g = (j * Hkv) // H
        s = (q[:, j, :] @ keys[:, g, :].T) * scale      # [T, S]
        s = np.where(mask, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        o[:, j, :] = p @ vals[:, g, :]
    return o


def chain_structure(t: int):
    """Depths and visibility of a linear block of t rows (row r sees rows 0..r)."""
    depth = np.arange(t, dtype=np.int64)
    vis = np.tril(np.ones((t, t), dtype=bool))
    return depth, vis


def tree_structure(parent):
    """Rows: 0 = pending token, row i+1 = draft node i with parent node parent[i]
    (-1 = the pending row).  Returns (depth[T], vis[T, T]) where vis[r, c] says
    block row c is an ancestor of row r or r itself."""
    parent = np.asarray(parent, dtype=np.int64)
    k = len(parent)
    t = k + 1
    prow = np.empty(t, dtype=np.int64)
    prow[0] = -1
    depth = np.zeros(t, dtype=np.int64)
    vis = np.zeros((t, t), dtype=bool)
    vis[0, 0] = True
    for i in range(k):
        p = int(parent[i])
        if not (-1 <= p < i):
            raise ValueError(f"parent[{i}] = {p} is not an earlier node")
        r = i + 1
        prow[r] = p + 1
        depth[r] = depth[p + 1] + 1
        vis[r] = vis[p + 1]
        vis[r, r] = True
    return depth, vis


def forward_block(shape, weights, cache, tokens, depth, vis, rounding_noise=None):
    """One forward of the target model over a block.

    shape   : model shape (n_layers, d_model, n_heads, n_kv_heads, head_dim,
              ffn, vocab, dtype, rms_eps, rope_theta)
    weights : object with .embed, .lm_head, .final_gain, .layer(l) -> mapping
              (wq, wk, wv, wo, w_gate, w_up, w_down, attn_gain, ffn_gain), arrays
              in the model dtype, logical [out, in] layout
    cache   : list per layer of (K, V), float64 [n, Hkv, hd] (already rounded)
    tokens  : [T] token ids; depth: [T]; vis: [T, T] bool
    rounding_noise : None (the definition above) or (generator, rel), a
              sensitivity probe for tests: every value rounded to bf16 is first
              multiplied by 1 + rel * N(0, 1), an error of the size a float32
              evaluation of the same expression carries.  The spread this
              causes in the logits is the part of a bf16 pipeline's result that
              its rounding points leave open (an operand within float32 error of
              a rounding boundary may round either way).
    Returns (logits [T, vocab] float64, block_kv: list per layer of (k, v) [T, Hkv, hd]).
    """
    dt = shape.dtype
    rnd = _rounder(dt)
    if rounding_noise is not None and dt == "bf16":
        gen, rel = rounding_noise
        exact = rnd

        def rnd(a):
            a = np.asarray(a, dtype=np.float64)
            return exact(a * (1.0 + rel * gen.standard_normal(a.shape)))
    H, Hkv, hd = shape.n_heads, shape.n_kv_heads, shape.head_dim
    tokens = np.asarray(tokens, dtype=np.int64)
    t = len(tokens)
    n = cache[0][0].shape[0] if cache else 0
    pos = n + np.asarray(depth, dtype=np.int64)
    scale = 1.0 / np.sqrt(hd)
    # visibility of [committed keys | block keys] for every row
    mask = np.concatenate([np.ones((t, n), dtype=bool), np.asarray(vis, dtype=bool)], axis=1)

    h = to_f64(weights.embed[tokens], dt)
    block_kv = []
    for l in range(shape.n_layers):
        lw = weights.layer(l)
        x = rnd(h * lw["attn_gain"].astype(np.float64))      # RMSNorm(h) * g = r * (h * g)
        r = norm_scale(h, shape.rms_eps)
        q = ((x @ to_f64(lw["wq"], dt).T) * r).reshape(t, H, hd)
        k = ((x @ to_f64(lw["wk"], dt).T) * r).reshape(t, Hkv, hd)
        v = ((x @ to_f64(lw["wv"], dt).T) * r).reshape(t, Hkv, hd)
        q = rnd(rope(q, pos, shape.rope_theta))
        k = rnd(rope(k, pos, shape.rope_theta))
        v = rnd(v)
        block_kv.append((k, v))
        kc, vc = cache[l] if cache else (np.zeros((0, Hkv, hd)), np.zeros((0, Hkv, hd)))
        keys = np.concatenate([kc, k], axis=0)          # [n + T, Hkv, hd]
        vals = np.concatenate([vc, v], axis=0)
        o = rnd(attention(q, keys, vals, mask, scale).reshape(t, H * hd))
        h = h + o @ to_f64(lw["wo"], dt).T
        x = rnd(h * lw["ffn_gain"].astype(np.float64))
        r = norm_scale(h, shape.rms_eps)
        z = rnd(silu((x @ to_f64(lw["w_gate"], dt).T) * r) * ((x @ to_f64(lw["w_up"], dt).T) * r))
        h = h + z @ to_f64(lw["w_down"], dt).T
    f = rnd(h * weights.final_gain.astype(np.float64))
    logits = (f @ to_f64(weights.lm_head, dt).T) * norm_scale(h, shape.rms_eps)
    return logits, block_kv
