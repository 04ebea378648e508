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
stores in bf16 are rounded to bf16 (nearest-even); the paper states no
precision, so these rounding sites are this implementation's reading of one
(the list is fixed; a kernel is checked against it, it does not follow a
kernel):

    x_attn   h * g_attn, the input of the q/k/v projections
    q, k     after RoPE (so the cache holds bf16 keys)
    v        the value projection (the cache holds bf16 values)
    o        the attention output, the input of the O projection
    x_ffn    h * g_ffn, the input of the gate/up projections
    z        silu(gate) * up, the input of the down projection
    x_final  h * g_final, the input of the LM head

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


ROUNDING_SITES = ("x_attn", "q", "k", "v", "o", "x_ffn", "z", "x_final")


def forward_block(shape, weights, cache, tokens, depth, vis, rounding=None):
    """One forward of the target model over a block.

    shape   : model shape (n_layers, d_model, n_heads, n_kv_heads, head_dim,
              ffn, vocab, dtype, rms_eps, rope_theta)
    weights : object with .embed, .lm_head, .final_gain, .layer(l) -> mapping
              (wq, wk, wv, wo, w_gate, w_up, w_down, attn_gain, ffn_gain), arrays
              in the model dtype, logical [out, in] layout
    cache   : list per layer of (K, V), float64 [n, Hkv, hd] (already rounded)
    tokens  : [T] token ids; depth: [T]; vis: [T, T] bool
    rounding: None (the definition above), or a test hook called at every
              rounding site of a bf16 model as rounding(site, layer, exact,
              rounded) with the site name (ROUNDING_SITES), the layer (n_layers
              for x_final), the exact float64 value and its bf16 rounding; the
              forward continues with what it returns.  Tests use it to probe
              the sensitivity to rounding flips, to drop one site, and to
              follow another evaluation's choice where a value lies so close
              to a bf16 rounding boundary that both neighbours are correct.
    Returns (logits [T, vocab] float64, block_kv: list per layer of (k, v) [T, Hkv, hd]).
    """
    dt = shape.dtype

    def rnd(site, layer, a):
        if dt != "bf16":
            return a
        r = round_bf16(a)
        return r if rounding is None else rounding(site, layer, a, r)

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
        x = rnd("x_attn", l, h * lw["attn_gain"].astype(np.float64))   # RMSNorm(h) * g = r * (h * g)
        r = norm_scale(h, shape.rms_eps)
        q = ((x @ to_f64(lw["wq"], dt).T) * r).reshape(t, H, hd)
        k = ((x @ to_f64(lw["wk"], dt).T) * r).reshape(t, Hkv, hd)
        v = ((x @ to_f64(lw["wv"], dt).T) * r).reshape(t, Hkv, hd)
        q = rnd("q", l, rope(q, pos, shape.rope_theta))
        k = rnd("k", l, rope(k, pos, shape.rope_theta))
        v = rnd("v", l, v)
        block_kv.append((k, v))
        kc, vc = cache[l] if cache else (np.zeros((0, Hkv, hd)), np.zeros((0, Hkv, hd)))
        keys = np.concatenate([kc, k], axis=0)          # [n + T, Hkv, hd]
        vals = np.concatenate([vc, v], axis=0)
        o = rnd("o", l, attention(q, keys, vals, mask, scale).reshape(t, H * hd))
        h = h + o @ to_f64(lw["wo"], dt).T
        x = rnd("x_ffn", l, h * lw["ffn_gain"].astype(np.float64))
        r = norm_scale(h, shape.rms_eps)
        z = rnd("z", l, silu((x @ to_f64(lw["w_gate"], dt).T) * r) * ((x @ to_f64(lw["w_up"], dt).T) * r))
        h = h + z @ to_f64(lw["w_down"], dt).T
    f = rnd("x_final", shape.n_layers, h * weights.final_gain.astype(np.float64))
    logits = (f @ to_f64(weights.lm_head, dt).T) * norm_scale(h, shape.rms_eps)
    return logits, block_kv
