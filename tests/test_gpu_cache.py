"""Content-addressed weight loading (wici_load_weights_cached) on the GPU: the
paper's model-caching exchange (hashes first, tensors only on a miss) through the
C ABI.  A model loaded from the store must match the float64 oracle (greedy ids
identical, logits within 2e-2 of the largest) and be bitwise equal to a plain
upload."""

from __future__ import annotations

import os

import numpy as np
import pytest

from paper_2608_24204_amd import configs, inputs
from tests.parity import compare, oracle_run

pytestmark = pytest.mark.gpu

CFG = configs.ModelConfig(name="t_cache", key=90, n_layers=2, d_model=512, n_heads=8,
                          n_kv_heads=2, head_dim=64, ffn_dim=1024, vocab=3001, prompt_len=40,
                          decode_steps=8)


def _run(m, prompt):
    ids, logs = m.generate(prompt, CFG.decode_steps, want_logits=True)
    return ids, np.stack(logs)


def test_cache_exchange_matches_plain_upload(cuda_ok, tmp_path):
    from paper_2608_24204_amd.binding import (WICI_CACHE_HIT, WICI_CACHE_NEEDED, WICI_CACHE_SAVED,
                                              WICI_CACHE_SENT, WICI_E_STATE, WiciError, WiciModel,
                                              md5)
    w = inputs.make_weights(CFG, gain_std=0.1)
    prompt = inputs.make_prompt(CFG)
    store = str(tmp_path / "store")
    os.makedirs(store)
    threshold = 300_000                        # the 3001 x 512 embedding and the MLP matrices
    big = {n for n, a in w.items() if a.nbytes >= threshold}
    assert big and len(big) < len(w)

    ref = WiciModel(CFG)
    try:
        ref.load_weights(w)
        ids0, lg0 = _run(ref, prompt)
    finally:
        ref.close()

    # cold store: everything sent, the large tensors saved under their MD5
    m1 = WiciModel(CFG)
    try:
        out = m1.load_weights_cached(w, store, threshold)
        assert {n for n, o in out.items() if o == WICI_CACHE_SAVED} == big
        assert all(o == WICI_CACHE_SENT for n, o in out.items() if n not in big)
        for n in big:
            path = os.path.join(store, md5(w[n]).hex())
            assert os.path.getsize(path) == w[n].nbytes
        ids1, lg1 = _run(m1, prompt)
    finally:
        m1.close()
    assert ids1 == ids0 and np.array_equal(lg1, lg0)

    # warm store, hashes only for the large tensors (sent without data): all hits
    hashes = {n: md5(w[n]) for n in big}
    m2 = WiciModel(CFG)
    try:
        out = m2.load_weights_cached(w, store, threshold, hashes=hashes)
        assert all(out[n] == WICI_CACHE_HIT for n in big)
        ids2, lg2 = _run(m2, prompt)
    finally:
        m2.close()
    assert ids2 == ids0 and np.array_equal(lg2, lg0)
    # the model loaded from the store against the oracle's own greedy run
    rep = compare(ids2, list(lg2), *oracle_run(CFG, inputs.weights_f64(CFG, w), prompt,
                                                CFG.decode_steps))
    print(f"[cache parity] {rep.summary()}", flush=True)
    assert rep.max_rel_err <= 2e-2
    assert rep.strict_ids, rep.summary()

    # one file missing and one of the wrong size: both needed; resend with data
    lost, bad = sorted(big)[:2]
    os.remove(os.path.join(store, hashes[lost].hex()))
    with open(os.path.join(store, hashes[bad].hex()), "r+b") as f:
        f.truncate(16)
    m3 = WiciModel(CFG)
    try:
        out = m3.load_weights_cached(w, store, threshold, hashes=hashes)
        assert out[lost] == WICI_CACHE_NEEDED and out[bad] == WICI_CACHE_NEEDED
        assert sum(o == WICI_CACHE_NEEDED for o in out.values()) == 2
        with pytest.raises(WiciError) as e:
            m3.prefill(prompt)                    # two tensors still missing
        assert e.value.status == WICI_E_STATE
        out = m3.load_weights_cached({lost: w[lost], bad: w[bad]}, store, threshold)
        assert out[lost] == WICI_CACHE_SAVED and out[bad] == WICI_CACHE_SAVED
        ids3, lg3 = _run(m3, prompt)
    finally:
        m3.close()
    assert ids3 == ids0 and np.array_equal(lg3, lg0)
    assert os.path.getsize(os.path.join(store, hashes[bad].hex())) == w[bad].nbytes
