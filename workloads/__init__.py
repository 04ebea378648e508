"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This module only *draws* inputs: model shapes, random weights, Zipf token
streams, edited copies of a token stream, random draft trees and planted
drafts.  It holds none of the verification method's arithmetic (no forward
pass, no argmax, no acceptance rule), so the CPU oracle and the GPU path can
both consume it without sharing any of the computation they are compared on.
"""

from .configs import CONFIGS, ModelShape, get_shape
from .weights import WeightSet, gen_weights, bf16_bits_to_f32
from .tokens import (zipf_tokens, inject_edits, random_tree, tree_tokens, planted_draft,
                     random_kv_context)

__all__ = [
    "CONFIGS", "ModelShape", "get_shape", "WeightSet", "gen_weights",
    "bf16_bits_to_f32", "zipf_tokens", "inject_edits", "random_tree", "tree_tokens",
    "planted_draft", "random_kv_context",
]
