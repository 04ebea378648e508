"""Model shapes of the synthetic Llama-style decoders used as verification targets.

The paper's target models (Qwen2.5-Coder-32B, DeepSeek-Coder-33B and their
7B/6.7B draft siblings; Implementation Details) are not available, so their
weights are replaced by random ones drawn from a seed.  The shapes below are
generic Llama-style decoders of the four sizes the measurements use.
"""

from dataclasses import dataclass, asdict, replace


@dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    dtype: str            # "f32" or "bf16": weights, KV cache and GEMM inputs
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def with_(self, **kw) -> "ModelShape":
        return replace(self, **kw)

    def asdict(self) -> dict:
        return asdict(self)


CONFIGS = {
    # 2 layers, fp32 end to end; the small case every parity test starts from.
    "tiny": ModelShape("tiny-f32", 2, 256, 4, 4, 64, 688, 1024, "f32"),
    "1b": ModelShape("llama-1b-bf16", 16, 2048, 16, 4, 128, 5632, 32256, "bf16"),
    "7b": ModelShape("llama-7b-bf16", 32, 4096, 32, 8, 128, 11008, 32256, "bf16"),
    "33b": ModelShape("llama-33b-bf16", 62, 7168, 56, 8, 128, 19200, 32256, "bf16"),
}


def get_shape(name: str, **overrides) -> ModelShape:
    s = CONFIGS[name]
    return s.with_(**overrides) if overrides else s
