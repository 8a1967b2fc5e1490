"""Full-size parity: a whole greedy request of each workload configuration (its
real shapes, prompt length and decode steps, in the launch configuration the
benchmark times) on the GPU, against the float64 oracle's own greedy run of the
same request.

The oracle's runs are stored in tests/golden/full/<config>.npz, written by
tests/golden/make_full_reference.py, which calls only the oracle and the seeded
input generator.  Each file keeps the oracle's ids and, per step, its largest
logit, its top 8 and 128 fixed sampled logits, plus the whole logit vector at
the prefill and at the last step.  A full-size float64 run takes minutes to over
ten minutes of host time (an 8192-token prompt, a 65 GB model).  The test checks
that the prompt and the weights are the ones the file was made from, then
compares (tests/parity.py, compare_fixture):
- strict: every generated id equals the oracle's;
- logits: at every step, max |g_i - o_i| / max |o_i| <= 2e-2 over the known
  entries (all of them at the two stored full vectors);
- wici_decode_n (the same steps device-resident in one call) gives the same ids.

Every configuration is held to the strict criterion except those listed in
NEAR_TIE: there the oracle's own margin at the named step is below what the
GPU's float32 arithmetic can resolve, so the test requires that the first
divergence is at that step and is a near tie by the two-token rule.  It
compares every step up to that one and prints the verdict as adjudicated.
"""

from __future__ import annotations

import json
import os
import time

import numpy as np
import pytest

from paper_2608_24204_amd import configs, inputs
from tests.parity import compare_fixture, load_fixture

pytestmark = pytest.mark.gpu

NAMES = ["1b", "8b", "8b_long", "32b", "1b_q8", "8b_q8", "32b_q8"]
# configuration -> the step of its recorded near tie: there the oracle's margin
# between its token and the GPU's (2.9e-3 for the 32B shape's 8-bit weights) is
# within twice the GPU's largest logit error away from those two tokens (8.2e-3
# to 9.6e-3 over the runs); the same step diverged in every run of the earlier
# kernels too
NEAR_TIE: dict[str, int] = {"32b_q8": 51}
TOL = 2e-2


def _report_path():
    d = os.path.join(os.environ.get("GRAFT_REPO_ROOT", "."), "gpurun_out")
    os.makedirs(d, exist_ok=True)
    return os.path.join(d, "full_parity.jsonl")


def _digests_match(fx, cfg, w, prompt):
    from tests.golden.make_full_reference import prompt_digest, weight_digest
    meta = fx["meta"]
    assert meta["config"] == cfg.name and meta["decode_steps"] == cfg.decode_steps
    assert meta["prompt_sha256"] == prompt_digest(prompt), "prompt differs from the stored run's"
    assert meta["weights_sha256"] == weight_digest(w), "weights differ from the stored run's"


@pytest.mark.parametrize("name", NAMES)
def test_full_size_greedy_run_matches_oracle(cuda_ok, name):
    from paper_2608_24204_amd.binding import WiciModel
    cfg = configs.CONFIGS[name]
    fx = load_fixture(name)
    t0 = time.time()
    w = inputs.make_weights(cfg)
    prompt = inputs.make_prompt(cfg)
    _digests_match(fx, cfg, w, prompt)
    print(f"[full parity] {name}: inputs ready ({time.time() - t0:.1f} s)", flush=True)
    m = WiciModel(cfg)
    try:
        m.load_weights(w)
        del w
        print(f"[full parity] {name}: weights loaded ({time.time() - t0:.1f} s)", flush=True)
        ids, logs = m.generate(prompt, cfg.decode_steps, want_logits=True)
        # the same request with the decode steps run device-resident in one call
        m.reset_kv()
        first, _ = m.prefill(prompt)
        toks, _ = m.decode_n(cfg.decode_steps)
        ids_n = [first] + [int(t) for t in toks]
    finally:
        m.close()
    rep = compare_fixture(ids, logs, fx)
    verdict = "strict" if rep.strict_ids else ("adjudicated" if rep.adjudicated else "failed")
    rec = {"config": name, "verdict": verdict, **rep.summary(),
           "near_tie_steps": rep.near_ties, "gpu_s": round(time.time() - t0, 1)}
    print("[full parity]", json.dumps(rec), flush=True)
    with open(_report_path(), "a") as f:
        f.write(json.dumps(rec) + "\n")
    assert rep.max_rel_err <= TOL, rec
    if name in NEAR_TIE:
        assert rep.strict_ids or (rep.first_divergence == NEAR_TIE[name] and rep.adjudicated), rec
    else:
        assert rep.strict_ids, rec
    assert ids_n == [int(i) for i in ids], "wici_decode_n differs from wici_decode_step"
