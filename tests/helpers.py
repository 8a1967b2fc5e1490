"""Small shared helpers for the tests (configs of test size, tolerance checks)."""

from __future__ import annotations

import numpy as np

from paper_2608_24204_amd.configs import ModelConfig


def small_cfg(**kw) -> ModelConfig:
    base = dict(name="small", key=50, n_layers=2, d_model=32, n_heads=4, n_kv_heads=2,
                head_dim=8, ffn_dim=48, vocab=64, weight_dtype="f32", kv_dtype="f32",
                prompt_len=12, decode_steps=6, rope_base=10000.0)
    base.update(kw)
    return ModelConfig(**base)


def inf_rel(a, b) -> float:
    """max_i |a_i - b_i| / max_i |b_i| (b is the reference)."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))
