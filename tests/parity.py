"""GPU-vs-oracle comparison of a greedy run (host logic shared by the GPU tests
and the benchmark's parity report).

Both sides run free: the oracle generates its own greedy ids from the prompt
(nothing from the GPU path goes into it), the GPU path its own.
- Token ids (strict): the two id sequences must be equal.
- Logits: at each step s where the contexts are still the same (every step up
  to and including the first divergence), max_i |g_i - o_i| / max_i |o_i| <= tol.
- Near ties: at the first step where the ids differ, let a be the oracle's token
  and b the GPU's.  The divergence counts as a near tie when the oracle's margin
  o_a - o_b is at most 2E.  E = max |g_i - o_i| over every index other than a
  and b: the error level of that step's GPU logits, measured away from the two
  tokens.  Errors of that size on a and b can swap them.  The two tokens' own
  errors cannot be the measure.  Whenever the GPU ranks b above a,
  |g_a - o_a| + |g_b - o_b| >= (g_b - g_a) + (o_a - o_b) >= o_a - o_b, so such
  a rule would call every divergence a near tie.  A near tie is reported, never
  counted as a pass of the strict criterion.  After it the contexts differ, so
  nothing later is compared.  `adjudicated` is the weaker verdict: strict, or
  the first divergence is a near tie.

Against a stored full-size run (tests/golden/full/*.npz, written by
tests/golden/make_full_reference.py from the oracle alone) the oracle's logits
are known at a sample of indices per step, at its top 8, and in full at the
steps the file lists.  The error is then taken over the known entries.
"""

from __future__ import annotations

import json
import os
from dataclasses import dataclass, field

import numpy as np

from oracle import DecoderOracle

FIXTURE_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "full")


def oracle_run(cfg, w64, prompt, n_steps, kv_round=None, chunk=None, max_seq=None):
    """The oracle's own greedy run: prefill ``prompt`` (in chunks of ``chunk``),
    then ``n_steps`` decode steps each fed its own argmax.  Returns (ids, logits)
    with n_steps + 1 entries."""
    prompt = np.asarray(prompt, np.int64)
    orc = DecoderOracle(cfg, w64, kv_round=kv_round,
                        max_seq=max_seq or len(prompt) + n_steps)
    return orc.generate(prompt, n_steps, chunk)


@dataclass
class ParityReport:
    steps: int
    strict_ids: bool
    first_divergence: int | None
    compared: int = 0
    near_ties: list = field(default_factory=list)
    max_rel_err: float = 0.0
    worst_step: int = -1
    min_margin: float = float("inf")
    divergent: int = 0
    sampled: bool = False

    @property
    def adjudicated(self) -> bool:
        return self.strict_ids or len(self.near_ties) == self.divergent

    def summary(self) -> dict:
        return {"steps": self.steps, "compared": self.compared, "strict_ids": self.strict_ids,
                "first_divergence": self.first_divergence, "divergent": self.divergent,
                "near_ties": len(self.near_ties), "adjudicated": self.adjudicated,
                "max_rel_err": self.max_rel_err, "worst_step": self.worst_step,
                "min_oracle_margin": self.min_margin, "sampled": self.sampled}


def near_tie(o_a: float, o_b: float, level: float):
    """(is a near tie, oracle margin o_a - o_b, budget 2 * level) for the oracle's
    token a and the GPU's token b, where ``level`` is the step's largest logit
    error away from a and b."""
    margin = float(o_a - o_b)
    budget = 2.0 * float(level)
    return margin <= budget, margin, budget


def _level_away(err: np.ndarray, idx: np.ndarray, a: int, b: int) -> float:
    """Largest of the errors ``err`` (at indices ``idx``) other than at a and b."""
    keep = (idx != a) & (idx != b)
    return float(np.max(err[keep])) if np.any(keep) else 0.0


def compare(gpu_ids, gpu_logits, ora_ids, ora_logits) -> ParityReport:
    """Free-running GPU ids/logits against the oracle's free-running ids/logits."""
    gpu_ids = [int(t) for t in gpu_ids]
    ora_ids = [int(t) for t in ora_ids]
    rep = ParityReport(steps=len(gpu_ids), strict_ids=gpu_ids == ora_ids, first_divergence=None)
    for s in range(min(len(gpu_ids), len(ora_ids))):
        o = np.asarray(ora_logits[s], np.float64)
        top2 = np.partition(o, -2)[-2:]
        rep.min_margin = min(rep.min_margin, float(top2[1] - top2[0]))
        g = None
        if gpu_logits is not None and gpu_logits[s] is not None:
            g = np.asarray(gpu_logits[s], np.float64)
            rel = float(np.max(np.abs(g - o)) / np.max(np.abs(o)))
            if rel > rep.max_rel_err:
                rep.max_rel_err, rep.worst_step = rel, s
        rep.compared = s + 1
        if gpu_ids[s] != ora_ids[s]:
            rep.first_divergence, rep.divergent = s, 1
            a, b = ora_ids[s], gpu_ids[s]
            if g is not None:
                level = _level_away(np.abs(g - o), np.arange(o.size), a, b)
                ok, margin, budget = near_tie(o[a], o[b], level)
                if ok:
                    rep.near_ties.append((s, margin, budget))
            break
    if rep.first_divergence is None and len(gpu_ids) != len(ora_ids):
        rep.first_divergence, rep.divergent = rep.compared, 1
    return rep


# ---------------------------------------------------------------- stored full runs

def fixture_path(name: str) -> str:
    return os.path.join(FIXTURE_DIR, f"{name}.npz")


def load_fixture(name: str) -> dict:
    with np.load(fixture_path(name), allow_pickle=False) as z:
        fx = {k: z[k] for k in z.files}
    fx["meta"] = json.loads(str(fx["meta"]))
    return fx


def compare_fixture(gpu_ids, gpu_logits, fx) -> ParityReport:
    """Free-running GPU ids/logits against a stored oracle run (see the module
    docstring for which oracle logits are known at each step)."""
    gpu_ids = [int(t) for t in gpu_ids]
    ora_ids = [int(t) for t in fx["ids"]]
    rep = ParityReport(steps=len(gpu_ids), strict_ids=gpu_ids == ora_ids, first_divergence=None,
                       sampled=True)
    sidx = fx["sample_idx"]
    full_at = {int(s): j for j, s in enumerate(fx["full_steps"])}
    for s in range(min(len(gpu_ids), len(ora_ids))):
        tv = fx["top_val"][s]
        rep.min_margin = min(rep.min_margin, float(tv[0] - tv[1]))
        known = {int(i): float(v) for i, v in zip(sidx, fx["sample_val"][s])}
        known.update({int(i): float(v) for i, v in zip(fx["top_idx"][s], tv)})
        g = None
        if gpu_logits is not None and gpu_logits[s] is not None:
            g = np.asarray(gpu_logits[s], np.float64)
            if s in full_at:
                idx = np.arange(g.size)
                errs = np.abs(g - fx["full_logits"][full_at[s]].astype(np.float64))
            else:
                idx = np.fromiter(known.keys(), np.int64)
                errs = np.abs(g[idx] - np.fromiter(known.values(), np.float64))
            rel = float(np.max(errs)) / float(fx["max_abs"][s])
            if rel > rep.max_rel_err:
                rep.max_rel_err, rep.worst_step = rel, s
        rep.compared = s + 1
        if gpu_ids[s] != ora_ids[s]:
            rep.first_divergence, rep.divergent = s, 1
            a, b = ora_ids[s], gpu_ids[s]
            ob = known.get(b)
            if ob is None and s in full_at:
                ob = float(fx["full_logits"][full_at[s]][b])
            if g is not None and ob is not None:
                ok, margin, budget = near_tie(known[a], ob, _level_away(errs, idx, a, b))
                if ok:
                    rep.near_ties.append((s, margin, budget))
            break
    if rep.first_divergence is None and len(gpu_ids) != len(ora_ids):
        rep.first_divergence, rep.divergent = rep.compared, 1
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
        from oracle import dequantize_q8, quantize_q8
        a = self._f32(self.w[name])
        if a.ndim == 2:
            q, d = quantize_q8(a)
            return dequantize_q8(q, d)
        return a.astype(np.float64)

    def __contains__(self, name):
        return name in self.w

    def keys(self):
        return self.w.keys()
