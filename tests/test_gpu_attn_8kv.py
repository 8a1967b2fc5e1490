"""Decode attention at the shapes of the 1B- and 8B-shaped workloads' heads (8 KV
heads, 4 query heads per KV head; head dimension 128 and 64), bf16 weights and
cache, against the float64 oracle's own greedy run.  Capacities give 4 and 32
splits (merged in the last split block of each head, in the same launch) and 33
(merged by the separate merge kernel); wici_decode_n gives the same ids, and a
graph replay equals eager launches bit for bit."""

from __future__ import annotations

import numpy as np
import pytest

from paper_2608_24204_amd import configs, inputs
from tests.parity import compare, oracle_run

pytestmark = pytest.mark.gpu

CFGS = {
    "hd128": configs.ModelConfig(name="t_kv8_128", key=98, n_layers=2, d_model=1024, n_heads=32,
                                 n_kv_heads=8, head_dim=128, ffn_dim=1536, vocab=3001,
                                 prompt_len=150, decode_steps=12, rope_base=500000.0),
    "hd64": configs.ModelConfig(name="t_kv8_64", key=99, n_layers=2, d_model=512, n_heads=32,
                                n_kv_heads=8, head_dim=64, ffn_dim=1024, vocab=2003,
                                prompt_len=77, decode_steps=12, tied_embeddings=True),
}


def _run(cfg, w, prompt, n, **kw):
    from paper_2608_24204_amd.binding import WiciModel
    m = WiciModel(cfg, kv_page=16, **kw)
    try:
        m.load_weights(w)
        ids, logs = m.generate(prompt, n, want_logits=True)
        m.reset_kv()
        first, _ = m.prefill(prompt)
        toks, _ = m.decode_n(n)
    finally:
        m.close()
    assert [first] + [int(t) for t in toks] == ids
    return ids, np.stack(logs)


@pytest.mark.parametrize("cap", [None, 2048, 2049], ids=["splits4", "splits32", "splits33"])
@pytest.mark.parametrize("name", list(CFGS))
def test_decode_attention_8_kv_heads(cuda_ok, name, cap):
    cfg = CFGS[name]
    w = inputs.make_weights(cfg, gain_std=0.1)
    P = cfg.prompt_len if cap is None else cap - cfg.decode_steps - 3
    prompt = inputs.make_prompt(cfg, P)
    kw = {} if cap is None else {"max_seq": cap}
    ids, lg = _run(cfg, w, prompt, cfg.decode_steps, **kw)
    rep = compare(ids, list(lg), *oracle_run(cfg, inputs.weights_f64(cfg, w), prompt,
                                              cfg.decode_steps))
    print(f"[8 kv heads] {name} P={P} cap={cap}: {rep.summary()}", flush=True)
    assert rep.max_rel_err <= 2e-2
    assert rep.strict_ids, rep.summary()


def test_decode_attention_8_kv_heads_graph_equals_eager(cuda_ok):
    cfg = CFGS["hd128"]
    w = inputs.make_weights(cfg, gain_std=0.1)
    prompt = inputs.make_prompt(cfg)
    a = _run(cfg, w, prompt, 8)
    b = _run(cfg, w, prompt, 8, graph=False)
    assert a[0] == b[0] and np.array_equal(a[1], b[1])


# Prefill attention with 32 query heads and a chunk whose query-block count does
# not divide the CU count: more (query block, head) pairs than CUs, so the
# long/short pairing of causal walks reverses the block order for some heads and
# not others, which must still cover every (head, query block) exactly once.
# The fp32-cache case runs the vector kernel, the bf16 ones the matrix-core one.
F32 = configs.ModelConfig(name="t_kv8_f32", key=97, n_layers=2, d_model=512, n_heads=32,
                          n_kv_heads=8, head_dim=64, ffn_dim=768, vocab=1009,
                          weight_dtype="f32", kv_dtype="f32", prompt_len=700, decode_steps=4)


@pytest.mark.parametrize("name,P,chunk", [("hd128", 700, None), ("hd128", 1000, 640),
                                          ("hd64", 700, None), ("f32", 700, None)])
def test_prefill_attention_many_heads_ragged_blocks(cuda_ok, name, P, chunk):
    cfg = F32 if name == "f32" else CFGS[name]
    w = inputs.make_weights(cfg, gain_std=0.1)
    prompt = inputs.make_prompt(cfg, P)
    kw = {"max_seq": P + 16} if chunk is None else {"max_seq": P + 16, "prefill_chunk": chunk}
    ids, lg = _run(cfg, w, prompt, 4, **kw)
    rep = compare(ids, list(lg), *oracle_run(cfg, inputs.weights_f64(cfg, w), prompt, 4))
    print(f"[prefill 32 heads] {name} P={P} chunk={chunk}: {rep.summary()}", flush=True)
    assert rep.max_rel_err <= (1e-4 if cfg.weight_dtype == "f32" else 2e-2)
    assert rep.strict_ids, rep.summary()
