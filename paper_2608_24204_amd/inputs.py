"""Seeded synthetic inputs (weights and prompt ids) shared by the GPU path, its
tests and the benchmark.

This module draws random numbers and stores them in the workload's storage
formats; it computes nothing of the forward pass itself.

Weights: every matrix and the embedding ~ N(0, 0.02^2), drawn in float32 from
numpy's PCG64 stream keyed by (weight_seed, config key, tensor index, block index)
over blocks of 2**24 elements, then rounded to the nearest bfloat16 (ties to even)
for bf16 configurations.  Norm gains are 1.0 unless ``gain_std`` asks for
1 + N(0, gain_std^2) (tests use random gains so that a gain applied to the wrong
vector is caught).  Prompt ids are uniform in [0, vocab) from the stream
(prompt_seed, config key).

bf16 tensors are returned as uint16 arrays holding the bf16 bit patterns; float32
tensors (norm gains, fp32 configurations) as float32 arrays.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .configs import ModelConfig

WEIGHT_SEED = 0
PROMPT_SEED = 1
INIT_STD = 0.02
BLOCK = 1 << 24


def tensor_specs(cfg: ModelConfig):
    """(name, shape, kind) in the fixed generation order; kind is 'mat' or 'gain'."""
    d, F, V = cfg.d_model, cfg.ffn_dim, cfg.vocab
    specs = [("tok_embeddings", (V, d), "mat")]
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        specs += [
            (p + "attn_norm", (d,), "gain"),
            (p + "wq", (cfg.q_dim, d), "mat"),
            (p + "wk", (cfg.kv_dim, d), "mat"),
            (p + "wv", (cfg.kv_dim, d), "mat"),
            (p + "wo", (d, cfg.q_dim), "mat"),
            (p + "ffn_norm", (d,), "gain"),
            (p + "w_gate", (F, d), "mat"),
            (p + "w_up", (F, d), "mat"),
            (p + "w_down", (d, F), "mat"),
        ]
    specs.append(("norm", (d,), "gain"))
    if not cfg.tied_embeddings:
        specs.append(("lm_head", (V, d), "mat"))
    return specs


def f32_to_bf16_bits(src: np.ndarray, out: np.ndarray) -> None:
    """Round float32 values to the nearest bfloat16 (ties to even); write the bit
    patterns into the uint16 array ``out`` (same number of elements)."""
    u = src.view(np.uint32).ravel()
    t = np.right_shift(u, 16)
    np.bitwise_and(t, 1, out=t)
    t += 0x7FFF
    t += u
    np.right_shift(t, 16, out=t)
    out.ravel()[:] = t


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def _fill_block(cfg, tidx, b, flat_out, is_bf16, seed):
    n = flat_out.size
    lo = b * BLOCK
    hi = min(n, lo + BLOCK)
    rng = np.random.default_rng([seed, cfg.key, tidx, b])
    buf = rng.standard_normal(hi - lo, dtype=np.float32)
    buf *= np.float32(INIT_STD)
    if is_bf16:
        f32_to_bf16_bits(buf, flat_out[lo:hi])
    else:
        flat_out[lo:hi] = buf


def make_weights(cfg: ModelConfig, seed: int = WEIGHT_SEED, gain_std: float = 0.0,
                 threads: int | None = None) -> dict[str, np.ndarray]:
    """All weight tensors of ``cfg`` by name (see module docstring for the recipe)."""
    is_bf16 = cfg.weight_dtype in ("bf16", "q8")   # q8 models start from bf16 weights
    out: dict[str, np.ndarray] = {}
    jobs = []
    for tidx, (name, shape, kind) in enumerate(tensor_specs(cfg)):
        if kind == "gain":
            if gain_std > 0:
                rng = np.random.default_rng([seed, cfg.key, tidx])
                g = 1.0 + gain_std * rng.standard_normal(shape, dtype=np.float32)
                out[name] = g.astype(np.float32)
            else:
                out[name] = np.ones(shape, np.float32)
            continue
        arr = np.empty(shape, np.uint16 if is_bf16 else np.float32)
        out[name] = arr
        nblk = (arr.size + BLOCK - 1) // BLOCK
        for b in range(nblk):
            jobs.append((tidx, b, arr.reshape(-1)))
    if threads is None:
        threads = min(16, os.cpu_count() or 1)
    if threads <= 1 or len(jobs) == 1:
        for tidx, b, flat in jobs:
            _fill_block(cfg, tidx, b, flat, is_bf16, seed)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(lambda j: _fill_block(cfg, j[0], j[1], j[2], is_bf16, seed), jobs))
    return out


def make_prompt(cfg: ModelConfig, n: int | None = None, seed: int = PROMPT_SEED) -> np.ndarray:
    n = cfg.prompt_len if n is None else n
    rng = np.random.default_rng([seed, cfg.key])
    return rng.integers(0, cfg.vocab, n).astype(np.int32)


def weights_f64(cfg: ModelConfig, weights: dict[str, np.ndarray],
                threads: int | None = None) -> dict[str, np.ndarray]:
    """The exact values of the stored weights as float64 arrays (storage decoding
    only: a bf16 bit pattern is widened, never re-rounded)."""
    is_bf16 = cfg.weight_dtype in ("bf16", "q8")   # q8 models start from bf16 weights

    def conv(item):
        name, a = item
        if a.dtype == np.uint16:
            assert is_bf16
            return name, bf16_bits_to_f32(a).astype(np.float64)
        return name, a.astype(np.float64)

    if threads is None:
        threads = min(16, os.cpu_count() or 1)
    with ThreadPoolExecutor(max(1, threads)) as ex:
        return dict(ex.map(conv, weights.items()))


class LazyF64:
    """Read-only mapping name -> float64 array that widens the stored weight on
    each access (nothing is cached), so a float64 forward over a model that is too
    large to hold in float64 touches one matrix at a time."""

    def __init__(self, weights: dict[str, np.ndarray]):
        self._w = weights

    def __getitem__(self, name: str) -> np.ndarray:
        a = self._w[name]
        if a.dtype == np.uint16:
            return bf16_bits_to_f32(a).astype(np.float64)
        return a.astype(np.float64)

    def __contains__(self, name: str) -> bool:
        return name in self._w

    def keys(self):
        return self._w.keys()
