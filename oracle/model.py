"""Plain float64 CPU forward of a dense decoder-only transformer.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports, links or runs this
file; it exists to say what the GPU path must compute, slowly and obviously.

What is computed.  The paper offloads an LLM's GPU work as one fixed group of calls
per generated token whose inputs follow from the token index (Sec. "Batching and
Trace Replay", trace replay); the work is autoregressive inference of dense
decoder-only models (Sec. "Experiment Setup", Tab. "model_conf").  The paper never
writes the layer out, so this file takes the standard pre-norm decoder it runs:

  x_i = E[t_i]                                   token embedding, position i >= 0
  per layer:
    u   = RMSNorm(x; g_attn)                     x / sqrt(mean(x^2) + eps) * g
    q,k,v = W_q u, W_k u, W_v u                  [Hq,hd], [Hkv,hd], [Hkv,hd]
    q,k <- RoPE(., i)                            rotate-half pairs (j, j+hd/2),
                                                 angle i * base^(-2j/hd)
    cache k, v                                   stored in the KV storage type
    a_h = sum_j softmax_j(q_h . K_j,g / sqrt(hd)) V_j,g  over j <= i, g = h // (Hq/Hkv)
    x  += W_o concat_h(a_h)
    w   = RMSNorm(x; g_ffn)
    x  += W_down( silu(W_gate w) * (W_up w) )    silu(z) = z / (1 + e^-z)
  logits = W_lm RMSNorm(x_last; g_final)         W_lm = E when embeddings are tied
  token  = argmax(logits), lowest index on exact ties

Readings where the definition leaves room: no biases, no QK-norm, no RoPE scaling;
the KV cache holds bf16 values when the workload stores it in bf16 (k after RoPE and
v are rounded to the nearest bf16, ties to even, at the point they are cached), and
exact values otherwise (``kv_round``).

Pins (tests marked "not gpu"): softmax sums and shift invariance, single-key
attention, a triple-loop attention, GQA against a library attention on repeated
heads, RoPE norm / identity / relative-position properties, the RMSNorm closed form,
incremental = recompute, chunked = one-shot, causality, a scalar-loop forward on a
tiny model, and the Llama implementation of the `transformers` library.
"""

from __future__ import annotations

import math
from typing import Mapping

import numpy as np


# ---------------------------------------------------------------------------
# elementary operations
# ---------------------------------------------------------------------------

def bf16_round(x: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value (8 significant bits, ties to even) of float64 input,
    returned as float64.  Handles the bf16 subnormal range (quantum 2^-133) and
    overflow to +-inf; NaN stays NaN."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                      # x = m * 2^e, 0.5 <= |m| < 1
    # the leading bit is worth 2^(e-1); 8 significant bits -> quantum 2^(e-8)
    qexp = np.maximum(e - 8, -133)
    q = np.ldexp(np.ones_like(x), qexp)
    r = np.rint(x / q) * q                  # np.rint rounds half to even
    r = np.where(x == 0, x, r)
    big = np.ldexp(np.float64(0x1FF), 119)  # (2 - 2^-8) * 2^127: halfway past max
    r = np.where(np.abs(r) >= big, np.copysign(np.inf, x), r)
    # values between max bf16 and the halfway point round to max bf16
    maxbf = np.ldexp(np.float64(0xFF), 120)
    r = np.where((np.abs(x) > maxbf) & (np.abs(x) < big), np.copysign(maxbf, x), r)
    return r


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """Root-mean-square normalisation over the last axis, times the gain vector."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def softmax(s: np.ndarray, axis: int = -1) -> np.ndarray:
    m = np.max(s, axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def rope_rotate(z: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """Rotary position embedding, rotate-half convention.

    z: [T, H, hd]; positions: [T].  For j < hd/2 the pair (z_j, z_{j+hd/2}) is
    rotated by the angle positions * base^(-2j/hd)."""
    T, H, hd = z.shape
    half = hd // 2
    j = np.arange(half, dtype=np.float64)
    inv_freq = base ** (-2.0 * j / hd)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]  # [T, half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    a, b = z[..., :half], z[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray, q_pos: np.ndarray,
           k_pos: np.ndarray) -> np.ndarray:
    """Causal grouped-query attention.

    q: [T, Hq, hd] queries at positions q_pos [T]; K, V: [n, Hkv, hd] keys/values at
    positions k_pos [n].  Query head h reads KV head h // (Hq // Hkv); query at
    position p sees keys at positions <= p.  Returns [T, Hq, hd]."""
    T, Hq, hd = q.shape
    n, Hkv, _ = K.shape
    group = Hq // Hkv
    out = np.empty_like(q)
    mask = k_pos[None, :] <= q_pos[:, None]                    # [T, n]
    scale = 1.0 / math.sqrt(hd)
    for h in range(Hq):
        g = h // group
        s = (q[:, h, :] @ K[:, g, :].T) * scale                # [T, n]
        s = np.where(mask, s, -np.inf)
        p = softmax(s, axis=-1)
        out[:, h, :] = p @ V[:, g, :]
    return out


def greedy(logits: np.ndarray) -> int:
    """Index of the largest logit, lowest index among exact ties (numpy argmax)."""
    if not np.all(np.isfinite(logits)):
        raise FloatingPointError("non-finite logits")
    return int(np.argmax(logits))


# ---------------------------------------------------------------------------
# the model
# ---------------------------------------------------------------------------

class DecoderOracle:
    """Incremental (KV-cached) float64 forward.

    cfg: any object with n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim,
    vocab, rms_eps, rope_base, tied_embeddings and kv_dtype.
    weights: mapping name -> float64 array holding the exact stored weight values
    (names: tok_embeddings, layers.{l}.{attn_norm,wq,wk,wv,wo,ffn_norm,w_gate,w_up,
    w_down}, norm, lm_head).  A mapping that decodes on access keeps memory bounded
    for very large models.
    kv_round: 'bf16' stores cached k/v rounded to bf16, 'none' keeps them exact;
    default follows cfg.kv_dtype.
    """

    def __init__(self, cfg, weights: Mapping[str, np.ndarray], kv_round: str | None = None,
                 max_seq: int | None = None):
        self.cfg = cfg
        self.w = weights
        if kv_round is None:
            kv_round = "bf16" if cfg.kv_dtype == "bf16" else "none"
        assert kv_round in ("bf16", "none")
        self.kv_round = kv_round
        self.max_seq = max_seq if max_seq is not None else getattr(cfg, "max_seq", 4096)
        self.reset()

    def reset(self) -> None:
        c = self.cfg
        self.pos = 0
        self.K = [np.zeros((self.max_seq, c.n_kv_heads, c.head_dim)) for _ in range(c.n_layers)]
        self.V = [np.zeros((self.max_seq, c.n_kv_heads, c.head_dim)) for _ in range(c.n_layers)]

    def _store(self, a: np.ndarray) -> np.ndarray:
        return bf16_round(a) if self.kv_round == "bf16" else a

    def _lm_name(self) -> str:
        return "tok_embeddings" if self.cfg.tied_embeddings else "lm_head"

    def _embed(self, tokens: np.ndarray) -> np.ndarray:
        """Rows of the embedding as float64 (a mapping with ``rows`` widens only
        those rows)."""
        if hasattr(self.w, "rows"):
            return np.asarray(self.w.rows("tok_embeddings", tokens), dtype=np.float64)
        return self.w["tok_embeddings"][tokens].astype(np.float64)

    def _proj(self, u: np.ndarray, name: str) -> np.ndarray:
        """u @ W^T for the weight matrix ``name`` ([out, in]).  A mapping with
        ``project`` computes the same float64 product from its stored weights."""
        if hasattr(self.w, "project"):
            return self.w.project(name, u)
        return u @ self.w[name].T

    def forward(self, tokens, all_logits: bool = False, first_row: int = 0,
                progress=None) -> np.ndarray:
        """Append ``tokens`` at the current position; return the logits of the last
        appended position ([vocab]) or, with all_logits, of appended rows
        first_row.. ([T - first_row, vocab]).  ``progress(layer)`` is called after
        each layer (long runs report liveness through it)."""
        c = self.cfg
        tokens = np.asarray(tokens, dtype=np.int64).reshape(-1)
        T = tokens.size
        if T < 1:
            raise ValueError("empty token list")
        if np.any(tokens < 0) or np.any(tokens >= c.vocab):
            raise ValueError("token id out of range")
        if self.pos + T > self.max_seq:
            raise ValueError("sequence capacity exceeded")
        p0 = self.pos
        positions = np.arange(p0, p0 + T)
        x = self._embed(tokens)                                     # [T, d]
        for l in range(c.n_layers):
            pre = f"layers.{l}."
            u = rms_norm(x, self.w[pre + "attn_norm"], c.rms_eps)
            q = self._proj(u, pre + "wq").reshape(T, c.n_heads, c.head_dim)
            k = self._proj(u, pre + "wk").reshape(T, c.n_kv_heads, c.head_dim)
            v = self._proj(u, pre + "wv").reshape(T, c.n_kv_heads, c.head_dim)
            q = rope_rotate(q, positions, c.rope_base)
            k = rope_rotate(k, positions, c.rope_base)
            self.K[l][p0:p0 + T] = self._store(k)
            self.V[l][p0:p0 + T] = self._store(v)
            n = p0 + T
            a = attend(q, self.K[l][:n], self.V[l][:n], positions, np.arange(n))
            x = x + self._proj(a.reshape(T, c.n_heads * c.head_dim), pre + "wo")
            wn = rms_norm(x, self.w[pre + "ffn_norm"], c.rms_eps)
            h = silu(self._proj(wn, pre + "w_gate")) * self._proj(wn, pre + "w_up")
            x = x + self._proj(h, pre + "w_down")
            if progress is not None:
                progress(l)
        self.pos = p0 + T
        rows = x[first_row:] if all_logits else x[-1:]
        logits = self._proj(rms_norm(rows, self.w["norm"], c.rms_eps), self._lm_name())
        return logits if all_logits else logits[0]

    # -- the calls of the offload boundary, in oracle form --------------------

    def prefill(self, tokens, chunk: int | None = None) -> np.ndarray:
        """Process a prompt (optionally in chunks); return the last row's logits."""
        tokens = np.asarray(tokens).reshape(-1)
        if chunk is None or chunk >= tokens.size:
            return self.forward(tokens)
        out = None
        for s in range(0, tokens.size, chunk):
            out = self.forward(tokens[s:s + chunk])
        return out

    def decode(self, token: int) -> np.ndarray:
        return self.forward([int(token)])

    def full(self, tokens) -> np.ndarray:
        """Logits of every position of ``tokens`` recomputed from an empty cache."""
        self.reset()
        return self.forward(tokens, all_logits=True)

    def generate(self, prompt, n_steps: int, chunk: int | None = None):
        """Greedy run: prefill, then n_steps decode steps.  Returns (ids, logits)
        with n_steps + 1 generated ids and their logit vectors."""
        self.reset()
        lg = self.prefill(prompt, chunk)
        ids, logs = [greedy(lg)], [lg]
        for _ in range(n_steps):
            lg = self.decode(ids[-1])
            ids.append(greedy(lg))
            logs.append(lg)
        return ids, logs

    def teacher_forced(self, prompt, ids, chunk: int | None = None):
        """Logits of each step when the generated ids are forced to ``ids``:
        entry 0 is the prefill's, entry s the logits after feeding ids[s-1]."""
        self.reset()
        logs = [self.prefill(prompt, chunk)]
        for t in ids[:-1]:
            logs.append(self.decode(t))
        return logs
