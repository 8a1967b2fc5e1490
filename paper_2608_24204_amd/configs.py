"""Model and run configurations for the offloaded decoder forward.

The paper treats the offloaded work as an opaque, fixed group of GPU calls that is
repeated once per generated token with only the input changing (Sec. "Batching and
Trace Replay", trace replay); the models it runs are dense decoder-only LLMs served
by llama.cpp (Sec. "Experiment Setup", Tab. "model_conf").  The shapes below are the
five synthetic workloads this library is measured on.  Where a field is not fixed by
the workload description it carries the reading noted beside it.
"""

from __future__ import annotations

import dataclasses
from dataclasses import dataclass


@dataclass(frozen=True)
class ModelConfig:
    name: str
    key: int                 # stream key for the seeded input generator
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rms_eps: float = 1e-5    # reading: the only value stated for any workload, used for all
    rope_base: float = 10000.0
    tied_embeddings: bool = False
    weight_dtype: str = "bf16"   # "bf16", "f32", or "q8" (bf16 source weights stored as
                                 # block-scaled 8-bit codes: 34 bytes per 32 weights)
    kv_dtype: str = "bf16"       # KV cache storage type
    prompt_len: int = 32
    decode_steps: int = 16
    prefill_chunk: int = 2048
    kv_page: int = 64

    # ---- derived -------------------------------------------------------------
    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def max_seq(self) -> int:
        # prefill emits token 1; decode step i processes position P+i-1
        return self.prompt_len + self.decode_steps

    @property
    def wbytes(self) -> float:
        return {"bf16": 2, "f32": 4, "q8": 34 / 32}[self.weight_dtype]

    @property
    def kvbytes(self) -> int:
        return 2 if self.kv_dtype == "bf16" else 4

    def layer_matrix_params(self) -> int:
        d, F = self.d_model, self.ffn_dim
        return (self.q_dim + 2 * self.kv_dim) * d + d * self.q_dim + 2 * F * d + d * F

    def n_params(self) -> int:
        """All parameters: matrices, norm gains and the (possibly tied) embedding."""
        p = self.vocab * self.d_model  # embedding
        p += self.n_layers * (self.layer_matrix_params() + 2 * self.d_model)
        p += self.d_model  # final norm
        if not self.tied_embeddings:
            p += self.vocab * self.d_model
        return p

    def decode_bytes_per_token(self, n_ctx: int) -> int:
        """Algorithmic HBM bytes one decode step must move at context length n_ctx
        (keys attended, new position included): every layer matrix and the LM head
        once, and the KV cache read once per KV head.  The new position's keys and
        values written (2 kv_dim per layer) and the activation vectors are left
        out: under 0.001% of the total at the benchmarked shapes."""
        w = (self.n_layers * self.layer_matrix_params() + self.vocab * self.d_model) * self.wbytes
        kv_read = n_ctx * self.n_layers * 2 * self.kv_dim * self.kvbytes
        return int(round(w)) + kv_read

    def prefill_flops(self, n_prompt: int | None = None) -> int:
        """Algorithmic flops of a prefill: projections of every prompt row, causal
        attention (scores and weighted values, self included) and the LM head of the
        last row."""
        P = self.prompt_len if n_prompt is None else n_prompt
        proj = 2 * P * self.layer_matrix_params() * self.n_layers
        attn = self.n_layers * 4 * self.n_heads * self.head_dim * (P * (P + 1) // 2)
        return proj + attn + 2 * self.vocab * self.d_model

    def with_(self, **kw) -> "ModelConfig":
        return dataclasses.replace(self, **kw)


TINY = ModelConfig(
    name="tiny", key=0, n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
    ffn_dim=1024, vocab=4096, rope_base=10000.0, weight_dtype="f32", kv_dtype="f32",
    prompt_len=32, decode_steps=16)

LLAMA_1B = ModelConfig(
    name="1b", key=1, n_layers=16, d_model=2048, n_heads=32, n_kv_heads=8, head_dim=64,
    ffn_dim=8192, vocab=128256, tied_embeddings=True,
    rope_base=500000.0,       # reading: not stated; the shape family's value
    prompt_len=512, decode_steps=256)

LLAMA_8B = ModelConfig(
    name="8b", key=2, n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
    ffn_dim=14336, vocab=128256, rope_base=500000.0, prompt_len=1024, decode_steps=256)

LLAMA_8B_LONG = LLAMA_8B.with_(name="8b_long", key=3, prompt_len=8192, decode_steps=128)

QWEN_32B = ModelConfig(
    name="32b", key=4, n_layers=64, d_model=5120, n_heads=40, n_kv_heads=8, head_dim=128,
    ffn_dim=27648, vocab=152064,
    rope_base=1000000.0,      # reading: not stated; the shape family's value
    prompt_len=2048, decode_steps=128)

# The same models with their matrices stored block-scaled in 8 bits (the paper's
# applications run quantised GGUF models of about 8.5 bits per weight); same keys,
# so the same bf16 source weights.
LLAMA_1B_Q8 = LLAMA_1B.with_(name="1b_q8", weight_dtype="q8")
LLAMA_8B_Q8 = LLAMA_8B.with_(name="8b_q8", weight_dtype="q8")
QWEN_32B_Q8 = QWEN_32B.with_(name="32b_q8", weight_dtype="q8")

CONFIGS = {c.name: c for c in (TINY, LLAMA_1B, LLAMA_8B, LLAMA_8B_LONG, QWEN_32B,
                               LLAMA_1B_Q8, LLAMA_8B_Q8, QWEN_32B_Q8)}


def reduced(cfg: ModelConfig, n_layers: int, key_offset: int = 100, **kw) -> ModelConfig:
    """Same per-layer shape with fewer layers (and optionally other overrides); used
    by tests that need a full-width layer at a size the oracle finishes quickly."""
    return cfg.with_(name=f"{cfg.name}_L{n_layers}", key=cfg.key + key_offset,
                     n_layers=n_layers, **kw)
