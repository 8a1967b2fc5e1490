"""Host logic of the GPU-vs-oracle comparison (tests/parity.py): the strict and
the adjudicated verdicts on hand-made logits, live and against a stored run."""

import json

import numpy as np

from tests.parity import compare, compare_fixture, near_tie


def _logits(top, second, v=8):
    o = np.zeros(v)
    o[top], o[second] = 1.0, 0.5
    return o


def test_identical_run_is_strict():
    ora = [_logits(3, 1), _logits(5, 2)]
    rep = compare([3, 5], [o.copy() for o in ora], [3, 5], ora)
    assert rep.strict_ids and rep.adjudicated and rep.divergent == 0
    assert rep.max_rel_err == 0.0 and rep.min_margin == 0.5 and rep.compared == 2


def test_near_tie_is_judged_by_the_error_away_from_the_two_tokens():
    o = _logits(3, 1)
    o[1] = 0.999                       # oracle margin 0.001 between tokens 3 and 1
    g = o.copy()
    g[1], g[3] = 1.0004, 0.9996        # the GPU swaps them
    g[6] = 6e-4                        # error level elsewhere 6e-4: 2 * 6e-4 >= 1e-3
    rep = compare([1], [g], [3], [o])
    assert not rep.strict_ids and rep.divergent == 1 and rep.first_divergence == 0
    assert rep.adjudicated and len(rep.near_ties) == 1
    s, margin, budget = rep.near_ties[0]
    assert s == 0 and abs(margin - 1e-3) < 1e-12 and abs(budget - 1.2e-3) < 1e-12
    g[6] = 4e-4                        # error elsewhere 4e-4: 8e-4 < 1e-3
    rep = compare([1], [g], [3], [o])
    assert not rep.adjudicated


def test_a_swap_with_no_error_elsewhere_is_not_a_near_tie():
    # the two tokens' own errors always cover the margin when the GPU ranks b
    # above a; the rule must not use them
    o = _logits(3, 1)
    g = o.copy()
    g[1], g[3] = 1.2, 1.0              # GPU prefers token 1; oracle margin 0.5
    rep = compare([1], [g], [3], [o])
    assert not rep.adjudicated and rep.max_rel_err > 0.5


def test_near_tie_rule():
    ok, margin, budget = near_tie(1.0, 0.999, 6e-4)
    assert ok and abs(margin - 1e-3) < 1e-12 and abs(budget - 1.2e-3) < 1e-12
    ok, _, _ = near_tie(1.0, 0.5, 0.2)
    assert not ok


def test_comparison_stops_at_the_first_divergence():
    ora = [_logits(3, 1), _logits(5, 2), _logits(6, 2)]
    gpu = [o.copy() for o in ora]
    gpu[2] = gpu[2] * 100               # after the divergence: not compared
    rep = compare([3, 2, 0], gpu, [3, 5, 6], ora)
    assert rep.first_divergence == 1 and rep.compared == 2 and rep.max_rel_err == 0.0


def test_exact_logits_wrong_id_is_not_adjudicated():
    o = _logits(3, 1)
    rep = compare([1], [o.copy()], [3], [o])
    assert not rep.strict_ids and not rep.adjudicated


def _fixture(ora_logits, full_steps=(0,), sample=(0, 2, 4)):
    ora_logits = [np.asarray(o, np.float64) for o in ora_logits]
    ids = np.array([int(np.argmax(o)) for o in ora_logits], np.int32)
    top_idx = np.array([np.lexsort((np.arange(o.size), -o))[:3] for o in ora_logits], np.int32)
    top_val = np.array([o[i] for o, i in zip(ora_logits, top_idx)])
    sidx = np.array(sample, np.int32)
    return {"meta": json.loads('{"config": "x"}'), "ids": ids,
            "max_abs": np.array([np.max(np.abs(o)) for o in ora_logits]),
            "top_idx": top_idx, "top_val": top_val, "sample_idx": sidx,
            "sample_val": np.array([o[sidx] for o in ora_logits]),
            "full_steps": np.array(full_steps, np.int32),
            "full_logits": np.array([ora_logits[s] for s in full_steps], np.float32)}


def test_fixture_compare_strict_and_sampled_error():
    ora = [_logits(3, 1), _logits(5, 2), _logits(6, 7)]
    fx = _fixture(ora)
    gpu = [o.copy() for o in ora]
    gpu[1][4] += 0.01                   # a sampled index at a sampled-only step
    gpu[1][7] += 0.3                    # an index the file does not know at that step
    rep = compare_fixture([3, 5, 6], gpu, fx)
    assert rep.strict_ids and rep.compared == 3
    assert abs(rep.max_rel_err - 0.01) < 1e-12 and rep.worst_step == 1
    gpu[0][7] += 0.05                   # step 0 is stored in full: every index counts
    rep = compare_fixture([3, 5, 6], gpu, fx)
    assert abs(rep.max_rel_err - 0.05) < 1e-6 and rep.worst_step == 0


def test_fixture_compare_near_tie_from_top_values():
    o = _logits(3, 1)
    o[1] = 0.999
    fx = _fixture([o], full_steps=())
    g = o.copy()
    g[1], g[3] = 1.0004, 0.9996
    g[2] = 6e-4                        # sampled index 2: error level 6e-4 away from 1, 3
    rep = compare_fixture([1], [g], fx)
    assert not rep.strict_ids and rep.adjudicated and rep.first_divergence == 0
    g[2] = 4e-4
    rep = compare_fixture([1], [g], fx)
    assert not rep.adjudicated
