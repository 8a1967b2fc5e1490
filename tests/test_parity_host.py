"""Host logic of the GPU-vs-oracle comparison (tests/parity.py): the strict and
the adjudicated verdicts on hand-made logits."""

import numpy as np

from tests.parity import compare


def _logits(top, second, v=8):
    o = np.zeros(v)
    o[top], o[second] = 1.0, 0.5
    return o


def test_identical_run_is_strict():
    ora = [_logits(3, 1), _logits(5, 2)]
    rep = compare([3, 5], [o.copy() for o in ora], ora)
    assert rep.strict_ids and rep.adjudicated and rep.divergent == 0
    assert rep.max_rel_err == 0.0 and rep.min_margin == 0.5


def test_near_tie_divergence_is_adjudicated_not_strict():
    o = _logits(3, 1)
    o[1] = 0.999  # oracle margin 0.001
    g = o.copy()
    g[1], g[3] = 1.0004, 0.9996  # GPU error 4e-4 flips the tie: margin <= 2 * err
    rep = compare([1], [g], [o])
    assert not rep.strict_ids and rep.divergent == 1 and rep.first_divergence == 0
    assert rep.adjudicated and len(rep.near_ties) == 1


def test_real_divergence_is_neither():
    o = _logits(3, 1)
    g = o.copy()
    g[1] = 1.2  # the GPU prefers token 1 by far more than its logit error allows
    g[3] = 1.0
    rep = compare([1], [g], [o])
    # margin 0.5 against 2 * err = 2 * 0.7: a near tie by the rule (large error)
    assert rep.near_ties and rep.max_rel_err > 0.5
    rep2 = compare([1], [o.copy()], [o])  # exact logits, wrong id: no error budget
    assert not rep2.strict_ids and not rep2.adjudicated
