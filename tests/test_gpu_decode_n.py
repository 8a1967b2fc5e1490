"""Device-resident multi-step decode (wici_decode_n) through the C ABI: its tokens
against the float64 oracle's greedy run, bit-identity with per-step decoding,
runs split at arbitrary points, teacher forcing, capacity, and a step whose
logits stop being finite part-way through a run."""

from __future__ import annotations

import numpy as np
import pytest

from paper_2608_24204_amd import configs, inputs
from tests.parity import compare, oracle_run

pytestmark = pytest.mark.gpu

CFG = configs.ModelConfig(name="t_dn", key=74, n_layers=2, d_model=512, n_heads=8, n_kv_heads=2,
                          head_dim=128, ffn_dim=1024, vocab=2003, prompt_len=45,
                          decode_steps=40, rope_base=500000.0)
CFG32 = configs.ModelConfig(name="t_dn32", key=75, n_layers=2, d_model=256, n_heads=4,
                            n_kv_heads=4, head_dim=64, ffn_dim=512, vocab=1000,
                            weight_dtype="f32", kv_dtype="f32", prompt_len=21, decode_steps=30)

_W = {}


def weights(cfg):
    if cfg not in _W:
        _W[cfg] = inputs.make_weights(cfg, gain_std=0.1)
    return _W[cfg]


def model(cfg, w=None, **kw):
    from paper_2608_24204_amd.binding import WiciModel
    m = WiciModel(cfg, **kw)
    m.load_weights(weights(cfg) if w is None else w)
    return m


def stepwise(m, prompt, n):
    m.reset_kv()
    ids = [m.prefill(prompt)[0]]
    lg = None
    for _ in range(n):
        t, lg = m.decode_step(-1, want_logits=True)
        ids.append(t)
    return ids, lg


@pytest.mark.parametrize("cfg", [CFG, CFG32], ids=["bf16_gqa", "f32_mha"])
def test_decode_n_matches_oracle_and_decode_step(cuda_ok, cfg):
    w = weights(cfg)
    prompt = inputs.make_prompt(cfg)
    n = cfg.decode_steps
    m = model(cfg, kv_page=16)
    try:
        ref_ids, ref_lg = stepwise(m, prompt, n)
        m.reset_kv()
        first, _ = m.prefill(prompt)
        toks, lg = m.decode_n(n, want_logits=True)
        assert m.position == len(prompt) + n
    finally:
        m.close()
    ids = [first] + [int(t) for t in toks]
    assert ids == ref_ids
    assert np.array_equal(lg, ref_lg)      # same graph, same inputs: bitwise
    ora_ids, ora = oracle_run(cfg, inputs.weights_f64(cfg, w), prompt, n)
    rep = compare(ids, None, ora_ids, ora)
    print(f"[decode_n] {cfg.name}: {rep.summary()}", flush=True)
    assert rep.strict_ids, rep.summary()


def test_decode_n_split_runs_and_teacher_forcing(cuda_ok):
    prompt = inputs.make_prompt(CFG)
    m = model(CFG)
    try:
        ref, _ = stepwise(m, prompt, 20)
        # 20 steps as 1 + 7 + 12, mixing the per-step call in
        m.reset_kv()
        ids = [m.prefill(prompt)[0]]
        ids.append(m.decode_step(-1)[0])
        ids += [int(t) for t in m.decode_n(7)[0]]
        ids += [int(t) for t in m.decode_n(12)[0]]
        assert ids == ref
        # teacher forcing: an explicit token starts the run
        m.reset_kv()
        m.prefill(prompt)
        a = [m.decode_step(11)[0]] + [m.decode_step(-1)[0] for _ in range(4)]
        m.reset_kv()
        m.prefill(prompt)
        b = [int(t) for t in m.decode_n(5, token_in=11)[0]]
        assert a == b
    finally:
        m.close()


def test_decode_n_graph_and_eager_agree(cuda_ok):
    prompt = inputs.make_prompt(CFG)
    out = []
    for graph in (True, False):
        m = model(CFG, graph=graph)
        try:
            m.prefill(prompt)
            out.append(m.decode_n(16, want_logits=True))
        finally:
            m.close()
    assert np.array_equal(out[0][0], out[1][0])
    assert np.array_equal(out[0][1], out[1][1])


def test_decode_n_errors(cuda_ok):
    from paper_2608_24204_amd.binding import (WICI_E_ARG, WICI_E_CAPACITY, WICI_E_STATE,
                                              WiciError)
    m = model(CFG, max_seq=60)
    try:
        with pytest.raises(WiciError) as e:
            m.decode_n(3)                      # before any prefill
        assert e.value.status == WICI_E_STATE
        m.prefill(list(range(50)))
        with pytest.raises(WiciError) as e:
            m.decode_n(11)                     # 50 + 11 > 60: nothing runs
        assert e.value.status == WICI_E_CAPACITY
        assert m.position == 50
        with pytest.raises(WiciError) as e:
            m.decode_n(0)
        assert e.value.status == WICI_E_ARG
        with pytest.raises(WiciError) as e:
            m.decode_n(2, token_in=CFG.vocab)
        assert e.value.status == WICI_E_ARG
        toks, _ = m.decode_n(10)               # exactly fills the capacity
        assert len(toks) == 10 and m.position == 60
        assert all(0 <= t < CFG.vocab for t in toks)
        with pytest.raises(WiciError) as e:
            m.decode_n(1)
        assert e.value.status == WICI_E_CAPACITY
    finally:
        m.close()


def test_decode_n_stops_at_non_finite_logits(cuda_ok):
    """Poison the embedding row of the token a clean run emits at step k: the run
    returns the k clean tokens, step k+1 fails, the rest are no-ops, and a reset
    sequence runs clean again."""
    from paper_2608_24204_amd.binding import WICI_E_NUMERIC, WICI_E_STATE, WiciError
    cfg = CFG
    prompt = inputs.make_prompt(cfg)
    m = model(cfg)
    try:
        clean, _ = stepwise(m, prompt, 30)
    finally:
        m.close()
    seen = set(int(t) for t in prompt)
    k = None
    for s in range(1, 25):                     # clean[s] = token emitted by decode step s
        if clean[s] not in seen and clean[s] not in clean[:s]:
            k = s
            break
        seen.add(clean[s])
    assert k is not None
    w = dict(weights(cfg))
    emb = w["tok_embeddings"].copy()
    emb[clean[k]] = 0x7FC0                     # bf16 NaN bit pattern
    w["tok_embeddings"] = emb
    m = model(cfg, w=w)
    try:
        first, _ = m.prefill(prompt)
        assert first == clean[0]
        with pytest.raises(WiciError) as e:
            m.decode_n(20)
        assert e.value.status == WICI_E_NUMERIC
        assert [int(t) for t in e.value.tokens] == clean[1:k + 1]
        assert m.position == len(prompt) + k + 1   # the failed step was appended
        with pytest.raises(WiciError) as e:
            m.decode_n(2)                          # nothing to feed back
        assert e.value.status == WICI_E_STATE
        # an explicit token runs again, but the failed position cached non-finite
        # keys and values, so the sequence keeps failing until it is reset
        restart = (clean[k] + 1) % cfg.vocab
        with pytest.raises(WiciError) as e:
            m.decode_n(1, token_in=restart)
        assert e.value.status == WICI_E_NUMERIC and len(e.value.tokens) == 0
        assert m.position == len(prompt) + k + 2
        m.reset_kv()
        assert m.prefill(prompt)[0] == clean[0]
        toks, _ = m.decode_n(k)
        assert [int(t) for t in toks] == clean[1:k + 1]
    finally:
        m.close()
