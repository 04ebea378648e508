"""Seeded random weights for the synthetic decoders.

Every tensor has its own PCG64 stream, keyed by the run seed and a fixed
integer spawn key, so any single tensor (say one layer of a 33B-shaped model
that does not fit in host memory) can be regenerated on its own:

    embed            spawn key (0,)
    layer l, tensor j (1, l, j)   j: 0 wq, 1 wk, 2 wv, 3 wo, 4 w_gate, 5 w_up, 6 w_down
    lm_head          (2,)
    layer l gain j   (3, l, j)    j: 0 attention-side norm, 1 FFN-side norm
    final norm gain  (4,)

Linear weights are N(0, std^2) (std = 0.02 unless a test asks for a larger
spread, which keeps a small random model's greedy output from collapsing onto
one repeated token) in the logical [out, in] layout.  bf16 models
hold them as bf16 bit patterns (uint16, round-to-nearest-even from the fp32
draw); fp32 models hold the fp32 draw.  Norm gains are fp32: all ones by
default, or 1 + 0.1 N(0,1) when ``gains="random"`` (used by tests so that a
dropped gain is visible).
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

from .configs import ModelShape

LAYER_TENSORS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")
STD = 0.02


def _rng(seed: int, key: tuple) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=key)))


def _f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def tensor_shape(shape: ModelShape, name: str) -> tuple:
    d, qd, kd, f = shape.d_model, shape.q_dim, shape.kv_dim, shape.ffn
    return {
        "embed": (shape.vocab, d), "lm_head": (shape.vocab, d),
        "wq": (qd, d), "wk": (kd, d), "wv": (kd, d), "wo": (d, qd),
        "w_gate": (f, d), "w_up": (f, d), "w_down": (d, f),
    }[name]


def draw_tensor(shape: ModelShape, seed: int, key: tuple, dims: tuple,
                std: float = STD) -> np.ndarray:
    """One linear weight: fp32 N(0, std^2), stored in the model's dtype."""
    g = _rng(seed, key)
    a = np.empty(dims, dtype=np.float32)
    g.standard_normal(out=a, dtype=np.float32)
    a *= np.float32(std)
    if shape.dtype == "bf16":
        return _f32_to_bf16_bits(a)
    return a


def draw_gain(shape: ModelShape, seed: int, key: tuple, gains: str) -> np.ndarray:
    if gains == "ones":
        return np.ones(shape.d_model, dtype=np.float32)
    g = _rng(seed, key)
    return (1.0 + 0.1 * g.standard_normal(shape.d_model)).astype(np.float32)


class LayerWeights(dict):
    """wq, wk, wv, wo, w_gate, w_up, w_down, attn_gain, ffn_gain."""

    __getattr__ = dict.__getitem__


class WeightSet:
    """Weights of one synthetic model; layers can be materialised lazily.

    ``layer(l)`` returns a cached ``LayerWeights`` if the set was built eagerly,
    else regenerates layer ``l`` from its own streams on every call.
    """

    def __init__(self, shape: ModelShape, seed: int, gains: str = "ones",
                 eager: bool = True, threads: int | None = None, std: float = STD):
        self.shape, self.seed, self.gains, self.std = shape, seed, gains, std
        self._threads = threads or min(16, os.cpu_count() or 1)
        self._layers = None
        keys = [("embed", (0,)), ("lm_head", (2,))]
        with ThreadPoolExecutor(self._threads) as ex:
            embed, lm_head = ex.map(
                lambda kv: draw_tensor(shape, seed, kv[1], tensor_shape(shape, kv[0]), std), keys)
            self.embed, self.lm_head = embed, lm_head
            self.final_gain = draw_gain(shape, seed, (4,), gains)
            if eager:
                self._layers = list(ex.map(self._make_layer, range(shape.n_layers)))

    def _make_layer(self, l: int, ex: ThreadPoolExecutor | None = None) -> LayerWeights:
        s = self.shape
        jobs = [(name, (1, l, j)) for j, name in enumerate(LAYER_TENSORS)]
        if ex is None:
            arrs = [draw_tensor(s, self.seed, k, tensor_shape(s, n), self.std) for n, k in jobs]
        else:
            arrs = list(ex.map(lambda nk: draw_tensor(s, self.seed, nk[1], tensor_shape(s, nk[0]),
                                                      self.std), jobs))
        lw = LayerWeights(zip(LAYER_TENSORS, arrs))
        lw["attn_gain"] = draw_gain(s, self.seed, (3, l, 0), self.gains)
        lw["ffn_gain"] = draw_gain(s, self.seed, (3, l, 1), self.gains)
        return lw

    def layer(self, l: int) -> LayerWeights:
        if self._layers is not None:
            return self._layers[l]
        with ThreadPoolExecutor(self._threads) as ex:
            return self._make_layer(l, ex)

    def nbytes(self) -> int:
        tot = self.embed.nbytes + self.lm_head.nbytes
        for l in range(self.shape.n_layers):
            lw = self.layer(l) if self._layers is not None else None
            if lw is None:
                esz = 2 if self.shape.dtype == "bf16" else 4
                tot += esz * sum(int(np.prod(tensor_shape(self.shape, n))) for n in LAYER_TENSORS)
            else:
                tot += sum(lw[n].nbytes for n in LAYER_TENSORS)
        return tot


def gen_weights(shape: ModelShape, seed: int = 1234, gains: str = "ones",
                eager: bool = True, threads: int | None = None, std: float = STD) -> WeightSet:
    return WeightSet(shape, seed, gains=gains, eager=eager, threads=threads, std=std)
