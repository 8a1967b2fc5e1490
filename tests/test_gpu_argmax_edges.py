"""Greedy argmax edge cases through the C ABI (reading: lowest index among exactly
equal maxima), on every entry point that picks a token: wici_prefill,
wici_decode_step, wici_decode_n and wici_decode_batch.  The vocabulary (3001) is
not a multiple of the LM-head GEMV's row group, of its grid or of any tile.

- Exact ties: LM-head row i is a copy of base row i mod 7, so every logit value
  occurs about 430 times, spread over all row groups and workgroups.  Identical
  rows give bit-identical logits on both sides: the GEMV's sum over a row does
  not depend on the row's index, and the oracle's stored-weight products take
  each row through the same C loop.  The winner must be the lowest index with
  the largest value, i.e. the winning base row itself (an index below 7).
- Maximum at the last index: every layer matrix is zero, so the residual stream
  stays the token's embedding, whose dimension 0 is 1.0 (the other dimensions
  ~N(0, 0.02^2)).  The LM head's only non-zero column is 0: 0.5 (i + 1) / V for
  i < V - 1 and 1.0 for i = V - 1.  The logits then rise with i and their unique
  maximum is at V - 1.

The expected ids are the float64 oracle's own greedy run on the same weights."""

from __future__ import annotations

import numpy as np
import pytest

from oracle import DecoderOracle
from oracle.native import StoredWeights
from paper_2608_24204_amd import configs, inputs

pytestmark = pytest.mark.gpu

CFG = configs.ModelConfig(name="t_argmax", key=97, n_layers=2, d_model=512, n_heads=8,
                          n_kv_heads=2, head_dim=128, ffn_dim=768, vocab=3001, prompt_len=37,
                          decode_steps=10, rope_base=500000.0)
BASE = 7


def _bf16(a):
    out = np.empty(np.shape(a), np.uint16)
    inputs.f32_to_bf16_bits(np.ascontiguousarray(a, np.float32), out)
    return out


def tie_weights():
    w = dict(inputs.make_weights(CFG, gain_std=0.1))
    w["lm_head"] = np.ascontiguousarray(w["lm_head"][:BASE][np.arange(CFG.vocab) % BASE])
    return w


def last_index_weights():
    w = dict(inputs.make_weights(CFG))
    for n, a in w.items():
        if n.startswith("layers.") and a.ndim == 2:
            w[n] = np.zeros_like(a)
    emb = inputs.bf16_bits_to_f32(w["tok_embeddings"]).copy()
    emb[:, 0] = 1.0
    w["tok_embeddings"] = _bf16(emb)
    lm = np.zeros((CFG.vocab, CFG.d_model), np.float32)
    lm[:, 0] = 0.5 * (np.arange(CFG.vocab) + 1) / CFG.vocab
    lm[-1, 0] = 1.0
    w["lm_head"] = _bf16(lm)
    return w


def prompts(n):
    rng = np.random.default_rng(11)
    return [rng.integers(0, CFG.vocab, CFG.prompt_len - 5 * b).astype(np.int32) for b in range(n)]


def oracle_ids(w, prompt):
    orc = DecoderOracle(CFG, StoredWeights(w), max_seq=len(prompt) + CFG.decode_steps)
    return orc.generate(prompt, CFG.decode_steps)


@pytest.mark.parametrize("kind", ["ties", "last_index"])
def test_argmax_edges_on_every_entry_point(cuda_ok, kind):
    from paper_2608_24204_amd.binding import WiciModel
    w = tie_weights() if kind == "ties" else last_index_weights()
    ps = prompts(3)
    expect = []
    for p in ps:
        ids, logs = oracle_ids(w, p)
        if kind == "ties":
            for t, o in zip(ids, logs):
                assert t < BASE                                   # the lowest of its copies
                assert np.all(o[t::BASE] == o[t])                 # exactly tied copies
                assert np.sum(o == o[t]) >= CFG.vocab // BASE
        else:
            assert all(t == CFG.vocab - 1 for t in ids)
        expect.append(ids)

    lead = WiciModel(CFG, kv_page=16)
    clients = [lead]
    try:
        lead.load_weights(w)
        clients += [WiciModel(CFG, kv_page=16, share_weights_of=lead) for _ in range(len(ps) - 1)]
        for b, p in enumerate(ps):
            m = clients[b]
            # wici_prefill + wici_decode_step, with the logits (the GPU's own ties)
            ids, logs = m.generate(p, CFG.decode_steps, want_logits=True)
            assert ids == expect[b], (kind, "decode_step", b)
            for t, g in zip(ids, logs):
                assert g[t] == np.max(g) and not np.any(g[:t] == g[t])
            # wici_decode_n
            m.reset_kv()
            first, _ = m.prefill(p)
            toks, _ = m.decode_n(CFG.decode_steps)
            assert [first] + [int(t) for t in toks] == expect[b], (kind, "decode_n", b)
            m.reset_kv()
        # wici_decode_batch: the three clients advance together
        got = [[c.prefill(p)[0]] for c, p in zip(clients, ps)]
        for _ in range(CFG.decode_steps):
            toks = WiciModel.decode_batch(clients)
            for b in range(len(ps)):
                got[b].append(int(toks[b]))
        for b in range(len(ps)):
            assert got[b] == expect[b], (kind, "decode_batch", b)
    finally:
        for c in clients[::-1]:
            c.close()
