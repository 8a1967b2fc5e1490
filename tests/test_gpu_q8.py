"""Block-scaled 8-bit weights through the C ABI: the HIP path (decode GEMV on the
codes, prefill on the matrix cores with per-block scales, or the vector product)
against the float64 oracle run on the oracle's own quantisation of the same bf16
weights.  Tolerances as for bf16 weights: logits max relative error (infinity
norm) 2e-2, greedy ids identical at every step."""

from __future__ import annotations

import numpy as np
import pytest

from paper_2608_24204_amd import configs, inputs
from oracle import q8_model_f64
from tests.parity import compare, oracle_run

pytestmark = pytest.mark.gpu

Q8 = {
    "gqa128": configs.ModelConfig(name="q_gqa128", key=80, n_layers=2, d_model=512, n_heads=8,
                                  n_kv_heads=2, head_dim=128, ffn_dim=1536, vocab=2500,
                                  weight_dtype="q8", prompt_len=150, decode_steps=12,
                                  rope_base=500000.0),
    "gqa64_tied": configs.ModelConfig(name="q_gqa64", key=81, n_layers=2, d_model=512, n_heads=8,
                                      n_kv_heads=2, head_dim=64, ffn_dim=1024, vocab=3001,
                                      weight_dtype="q8", prompt_len=77, decode_steps=12,
                                      tied_embeddings=True),
    "g5": configs.ModelConfig(name="q_g5", key=82, n_layers=1, d_model=640, n_heads=10,
                              n_kv_heads=2, head_dim=128, ffn_dim=1536, vocab=1531,
                              weight_dtype="q8", prompt_len=33, decode_steps=8, rope_base=1e6),
}


def run(cfg, mode, **kw):
    from paper_2608_24204_amd.binding import WiciModel
    w = inputs.make_weights(cfg, gain_std=0.1)
    prompt = inputs.make_prompt(cfg)
    m = WiciModel(cfg, prefill_mode=mode, **kw)
    try:
        m.load_weights(w)
        ids, logs = m.generate(prompt, cfg.decode_steps, want_logits=True)
    finally:
        m.close()
    ora_ids, ora = oracle_run(cfg, q8_model_f64(w), prompt, cfg.decode_steps)
    rep = compare(ids, logs, ora_ids, ora)
    print(f"[q8 parity] {cfg.name} mode={mode} {kw} -> {rep.summary()}", flush=True)
    return rep


@pytest.mark.parametrize("mode", ["bf16x3q", "bf16x3", "f32"])
@pytest.mark.parametrize("name", list(Q8))
def test_q8_small_configs_match_oracle(cuda_ok, name, mode):
    rep = run(Q8[name], mode, kv_page=16)
    assert rep.max_rel_err <= 2e-2
    assert rep.strict_ids, rep.summary()


def test_q8_ragged_prompt_and_chunks(cuda_ok):
    cfg = Q8["gqa128"].with_(prompt_len=97)
    rep = run(cfg, "bf16x3", prefill_chunk=40, kv_page=32)
    assert rep.max_rel_err <= 2e-2
    assert rep.strict_ids, rep.summary()


def test_q8_decode_n_and_graph_agree(cuda_ok):
    from paper_2608_24204_amd.binding import WiciModel
    cfg = Q8["gqa64_tied"]
    w = inputs.make_weights(cfg, gain_std=0.1)
    prompt = inputs.make_prompt(cfg)
    out = []
    for graph in (True, False):
        m = WiciModel(cfg, graph=graph)
        try:
            m.load_weights(w)
            first, _ = m.prefill(prompt)
            toks, lg = m.decode_n(10, want_logits=True)
            out.append(([first] + [int(t) for t in toks], lg))
        finally:
            m.close()
    assert out[0][0] == out[1][0]
    assert np.array_equal(out[0][1], out[1][1])


def test_q8_rejects_non_finite_weights(cuda_ok):
    from paper_2608_24204_amd.binding import WICI_E_ARG, WiciError, WiciModel
    cfg = Q8["g5"]
    w = dict(inputs.make_weights(cfg))
    bad = w["layers.0.w_up"].copy()
    bad[3, 7] = 0x7F80                                   # bf16 +inf
    w["layers.0.w_up"] = bad
    m = WiciModel(cfg)
    try:
        with pytest.raises(WiciError) as e:
            m.load_weights(w)
        assert e.value.status == WICI_E_ARG
    finally:
        m.close()
