"""GPU-vs-oracle comparison of a greedy run (host logic shared by the GPU tests
and the benchmark's parity report).

Token ids: the GPU's free-running ids must equal, step by step, the argmax of the
oracle's logits computed with the same ids fed back (teacher forcing); up to the
first divergence this is the same as comparing two free-running sequences.
Logits: per step, max_i |g_i - o_i| / max_i |o_i| <= tol.
Near ties: at a step whose ids differ, the divergence is called a near tie when
the oracle's own margin between its token and the GPU's token is within twice the
largest logit error of that step (both tokens are then defensible); it is
reported, never counted as a pass of the strict criterion.  `adjudicated` is the
weaker verdict: every divergent step is such a near tie.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from oracle import DecoderOracle, dequantize_q8, quantize_q8


def oracle_step_logits(cfg, w64, prompt, ids, kv_round=None) -> np.ndarray:
    """Teacher-forced oracle logits for every generated step: row s is the logits
    the oracle produces after the prompt and ids[:s] (row 0 is the prefill's)."""
    prompt = np.asarray(prompt, np.int64)
    seq = np.concatenate([prompt, np.asarray(ids[:-1], np.int64)])
    orc = DecoderOracle(cfg, w64, kv_round=kv_round, max_seq=max(len(seq), 1))
    return orc.forward(seq, all_logits=True, first_row=len(prompt) - 1)


@dataclass
class ParityReport:
    steps: int
    strict_ids: bool
    first_divergence: int | None
    near_ties: list = field(default_factory=list)
    max_rel_err: float = 0.0
    worst_step: int = -1
    min_margin: float = float("inf")
    divergent: int = 0

    @property
    def adjudicated(self) -> bool:
        return len(self.near_ties) == self.divergent

    def summary(self) -> dict:
        return {"steps": self.steps, "strict_ids": self.strict_ids,
                "first_divergence": self.first_divergence, "divergent": self.divergent,
                "near_ties": len(self.near_ties), "adjudicated": self.adjudicated,
                "max_rel_err": self.max_rel_err, "min_oracle_margin": self.min_margin}


def compare(gpu_ids, gpu_logits, ora_logits) -> ParityReport:
    gpu_ids = list(gpu_ids)
    rep = ParityReport(steps=len(gpu_ids), strict_ids=True, first_divergence=None)
    for s, o in enumerate(ora_logits):
        top2 = np.partition(o, -2)[-2:]
        rep.min_margin = min(rep.min_margin, float(top2[1] - top2[0]))
        otok = int(np.argmax(o))
        err = None
        if gpu_logits is not None and gpu_logits[s] is not None:
            g = np.asarray(gpu_logits[s], np.float64)
            diff = np.abs(g - o)
            rel = float(diff.max() / np.abs(o).max())
            if rel > rep.max_rel_err:
                rep.max_rel_err, rep.worst_step = rel, s
            err = float(diff.max())
        if otok != gpu_ids[s]:
            if rep.first_divergence is None:
                rep.first_divergence = s
            rep.strict_ids = False
            rep.divergent += 1
            margin = float(o[otok] - o[gpu_ids[s]])
            if err is not None and margin <= 2 * err:
                rep.near_ties.append((s, margin, 2 * err))
    return rep


class LazyQ8F64:
    """Oracle weights of a block-scaled 8-bit model: each matrix (bf16 bits or
    float32) quantised by the oracle's own rule and dequantised to float64 when
    first asked for (norm gains are passed through); one tensor at a time, so a
    full-size model fits in host memory."""

    def __init__(self, weights):
        self.w = weights

    def _f32(self, a):
        a = np.asarray(a)
        if a.dtype == np.uint16:
            return (a.astype(np.uint32) << 16).view(np.float32)
        return a.astype(np.float32)

    def __getitem__(self, name):
        a = self._f32(self.w[name])
        if a.ndim == 2:
            q, d = quantize_q8(a)
            return dequantize_q8(q, d)
        return a.astype(np.float64)

    def __contains__(self, name):
        return name in self.w

    def keys(self):
        return self.w.keys()
