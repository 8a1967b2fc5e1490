"""Several clients on one GPU (wici_bind_memory_shared) and the batched decode
step (wici_decode_batch) through the C ABI: every sequence of a batch against the
float64 oracle (greedy ids identical at every step, logits within 2e-2 for bf16
weights and 1e-4 for fp32), and against the same sequence decoded alone."""

from __future__ import annotations

import numpy as np
import pytest

from oracle import DecoderOracle
from paper_2608_24204_amd import configs, inputs
from tests.parity import compare, oracle_run

pytestmark = pytest.mark.gpu

CFGS = {
    "bf16": configs.ModelConfig(name="t_batch", key=95, n_layers=2, d_model=512, n_heads=8,
                                n_kv_heads=2, head_dim=128, ffn_dim=1024, vocab=2003,
                                prompt_len=60, decode_steps=10, rope_base=500000.0),
    "f32": configs.ModelConfig(name="t_batch32", key=96, n_layers=2, d_model=256, n_heads=4,
                               n_kv_heads=4, head_dim=64, ffn_dim=512, vocab=1000,
                               weight_dtype="f32", kv_dtype="f32", prompt_len=30,
                               decode_steps=10),
}


def clients(cfg, w, n, **kw):
    from paper_2608_24204_amd.binding import WiciModel
    lead = WiciModel(cfg, **kw)
    lead.load_weights(w)
    return [lead] + [WiciModel(cfg, share_weights_of=lead, **kw) for _ in range(n - 1)]


def prompts(cfg, n):
    rng = np.random.default_rng(7)
    return [rng.integers(0, cfg.vocab, cfg.prompt_len - 9 * b).astype(np.int32) for b in range(n)]


@pytest.mark.parametrize("cap", [None, 5000], ids=["cap_default", "cap5000"])
@pytest.mark.parametrize("kind", list(CFGS))
def test_batched_decode_matches_oracle_per_sequence(cuda_ok, kind, cap):
    """cap5000: a capacity above 2048 positions, where each decode-attention
    block walks several 64-position sub-chunks."""
    cfg = CFGS[kind]
    w = inputs.make_weights(cfg, gain_std=0.1)
    w64 = inputs.weights_f64(cfg, w)
    tol = 1e-4 if cfg.weight_dtype == "f32" else 2e-2
    n = 4
    ps = prompts(cfg, n)
    ms = clients(cfg, w, n, kv_page=16, **({"max_seq": cap} if cap else {}))
    try:
        ids = [[] for _ in range(n)]
        logs = [[] for _ in range(n)]
        for b, m in enumerate(ms):
            t, lg = m.prefill(ps[b], want_logits=True)
            ids[b].append(t)
            logs[b].append(lg)
        for _ in range(cfg.decode_steps):
            toks, lg = ms[0].decode_batch(ms, want_logits=True)
            for b in range(n):
                ids[b].append(int(toks[b]))
                logs[b].append(lg[b])
        assert all(m.position == len(p) + cfg.decode_steps for m, p in zip(ms, ps))
    finally:
        for m in ms:
            m.close()
    for b in range(n):
        rep = compare(ids[b], logs[b], *oracle_run(cfg, w64, ps[b], cfg.decode_steps))
        print(f"[batch] {kind} seq {b} (P={len(ps[b])}): {rep.summary()}", flush=True)
        assert rep.max_rel_err <= tol
        assert rep.strict_ids, rep.summary()


@pytest.mark.parametrize("n,cap", [(20, 140), (33, 140), (8, 16384)])
def test_large_batches_match_oracle(cuda_ok, n, cap):
    """17-32 sequences: the batched products take the rows in two 16-row tiles
    (split along K for the projections with few weight rows, summed in the
    launch); past 32 they are the prefill's matrix-core products.  8 sequences
    at a 16384-position capacity (256 splits): the attention grid is past the
    size where the attention applies RoPE and appends itself, so the separate
    RoPE + append pass runs."""
    cfg = CFGS["bf16"]
    w = inputs.make_weights(cfg, gain_std=0.1)
    w64 = inputs.weights_f64(cfg, w)
    steps = 5
    rng = np.random.default_rng(11)
    ps = [rng.integers(0, cfg.vocab, 20 + 3 * b).astype(np.int32) for b in range(n)]
    ms = clients(cfg, w, n, kv_page=16, max_seq=cap)
    try:
        ids = [[m.prefill(p)[0]] for m, p in zip(ms, ps)]
        logs = [[] for _ in range(n)]
        for _ in range(steps):
            toks, lg = ms[0].decode_batch(ms, want_logits=True)
            for b in range(n):
                ids[b].append(int(toks[b]))
                logs[b].append(lg[b])
    finally:
        for m in ms:
            m.close()
    for b in range(n):
        ora_ids, ora = oracle_run(cfg, w64, ps[b], steps)
        # the prefill's logits are not compared here: only the batched steps
        rep = compare(ids[b], [None] + logs[b], ora_ids, ora)
        print(f"[batch] n={n} seq {b} (P={len(ps[b])}): {rep.summary()}", flush=True)
        assert rep.max_rel_err <= 2e-2
        assert rep.strict_ids, rep.summary()


def test_shared_weights_and_batch_agree_with_single_decoding(cuda_ok):
    from paper_2608_24204_amd.binding import WiciModel
    cfg = CFGS["bf16"]
    w = inputs.make_weights(cfg, gain_std=0.1)
    n = 3
    ps = prompts(cfg, n)
    # each sequence alone on its own model
    alone = []
    for b in range(n):
        m = WiciModel(cfg, max_seq=cfg.max_seq + 4)
        try:
            m.load_weights(w)
            ids, logs = m.generate(ps[b], cfg.decode_steps, want_logits=True)
            alone.append((ids, np.stack(logs)))
        finally:
            m.close()
    ms = clients(cfg, w, n, max_seq=cfg.max_seq + 4)
    try:
        # a shared-weight client decoding on its own is bitwise the same as alone
        ids, logs = ms[2].generate(ps[2], cfg.decode_steps, want_logits=True)
        assert ids == alone[2][0] and np.array_equal(np.stack(logs), alone[2][1])
        ms[2].reset_kv()
        got = [[m.prefill(p)[0]] for m, p in zip(ms, ps)]
        for _ in range(cfg.decode_steps):
            toks, lg = ms[0].decode_batch(ms, want_logits=True)
            for b in range(n):
                got[b].append(int(toks[b]))
        for b in range(n):
            assert got[b] == alone[b][0]
            # the batch's matrix products and the per-token GEMVs round differently
            ref = alone[b][1][-1]
            assert np.max(np.abs(lg[b] - ref)) <= 1e-3 * np.max(np.abs(ref))
        # batch of one, and explicit input tokens (teacher forcing)
        t1 = ms[0].decode_batch(ms[:1], tokens_in=[5])
        ms[0].reset_kv()
        ms[0].prefill(ps[0])
        for _ in range(cfg.decode_steps):
            ms[0].decode_step(-1)
        t2, _ = ms[0].decode_step(5)
        assert int(t1[0]) == t2
    finally:
        for m in ms:
            m.close()


def test_batch_errors(cuda_ok):
    from paper_2608_24204_amd.binding import (WICI_E_ARG, WICI_E_CAPACITY, WICI_E_STATE,
                                              WiciError, WiciModel)
    cfg = CFGS["bf16"]
    w = inputs.make_weights(cfg)
    ms = clients(cfg, w, 2, max_seq=70)
    other = WiciModel(cfg, max_seq=70)
    try:
        other.load_weights(w)
        with pytest.raises(WiciError) as e:
            ms[0].decode_batch(ms)                        # not prefilled
        assert e.value.status == WICI_E_STATE
        ms[0].prefill(list(range(69)))
        ms[1].prefill(list(range(10)))
        other.prefill(list(range(10)))
        with pytest.raises(WiciError) as e:
            ms[0].decode_batch([ms[0], ms[0]])            # duplicate
        assert e.value.status == WICI_E_ARG
        with pytest.raises(WiciError) as e:
            ms[0].decode_batch([ms[0], other])            # different weight copy
        assert e.value.status == WICI_E_ARG
        with pytest.raises(WiciError) as e:
            ms[1].load_weights(w)                         # shared weights are read-only
        assert e.value.status == WICI_E_STATE
        toks = ms[0].decode_batch(ms)                     # ms[0] reaches 70 = max_seq
        assert len(toks) == 2
        with pytest.raises(WiciError) as e:
            ms[0].decode_batch(ms)
        assert e.value.status == WICI_E_CAPACITY
        with pytest.raises(WiciError) as e:
            WiciModel(cfg.with_(d_model=256), share_weights_of=ms[0])
        assert e.value.status == WICI_E_ARG
    finally:
        for m in ms + [other]:
            m.close()


def test_fault_drill_fails_the_batched_step(cuda_ok):
    """WICI_FLAG_FAULT_DRILL on the lead: every split-K sum of the batched
    products reports its splits as run on different XCDs, so the step fails
    with WICI_E_HIP and the lead stays failed (the path a real misplacement
    takes; the kernels run normally)."""
    from paper_2608_24204_amd.binding import WICI_E_HIP, WICI_E_STATE, WiciError, WiciModel
    cfg = CFGS["bf16"]
    w = inputs.make_weights(cfg)
    lead = WiciModel(cfg, max_seq=80, fault_drill=True)
    ms = [lead]
    try:
        lead.load_weights(w)
        ms.append(WiciModel(cfg, max_seq=80, share_weights_of=lead))
        for m, p in zip(ms, prompts(cfg, 2)):
            m.prefill(p)
        with pytest.raises(WiciError) as e:
            lead.decode_batch(ms)
        assert e.value.status == WICI_E_HIP and "XCD" in str(e.value)
        with pytest.raises(WiciError) as e:
            lead.decode_batch(ms)
        assert e.value.status == WICI_E_STATE
    finally:
        for m in ms:
            m.close()


GROUP_CFGS = {
    "hd64_g4": configs.ModelConfig(name="t_batch_hd64", key=97, n_layers=2, d_model=512, n_heads=8,
                                   n_kv_heads=2, head_dim=64, ffn_dim=1024, vocab=1500,
                                   prompt_len=40, decode_steps=6, rope_base=500000.0),
    "hd128_g5": configs.ModelConfig(name="t_batch_g5", key=98, n_layers=2, d_model=640,
                                    n_heads=10, n_kv_heads=2, head_dim=128, ffn_dim=1536,
                                    vocab=1531, prompt_len=40, decode_steps=6, rope_base=1e6),
    "hd128_g8": configs.ModelConfig(name="t_batch_g8", key=99, n_layers=2, d_model=512,
                                    n_heads=16, n_kv_heads=2, head_dim=128, ffn_dim=1024,
                                    vocab=1700, prompt_len=40, decode_steps=6),
}


@pytest.mark.parametrize("name", list(GROUP_CFGS))
def test_batched_attention_shapes_match_oracle(cuda_ok, name):
    """The batched attention with its own RoPE + append at head dimension 64
    (each RoPE pair in one lane's steps 0 and 1) and with 5 and 8 query heads
    per KV head."""
    cfg = GROUP_CFGS[name]
    w = inputs.make_weights(cfg, gain_std=0.1)
    w64 = inputs.weights_f64(cfg, w)
    n = 3
    rng = np.random.default_rng(5)
    ps = [rng.integers(0, cfg.vocab, cfg.prompt_len - 7 * b).astype(np.int32) for b in range(n)]
    ms = clients(cfg, w, n, kv_page=16, max_seq=cfg.prompt_len + cfg.decode_steps + 2)
    try:
        ids = [[m.prefill(p)[0]] for m, p in zip(ms, ps)]
        logs = [[] for _ in range(n)]
        for _ in range(cfg.decode_steps):
            toks, lg = ms[0].decode_batch(ms, want_logits=True)
            for b in range(n):
                ids[b].append(int(toks[b]))
                logs[b].append(lg[b])
    finally:
        for m in ms:
            m.close()
    for b in range(n):
        ora_ids, ora = oracle_run(cfg, w64, ps[b], cfg.decode_steps)
        rep = compare(ids[b], [None] + logs[b], ora_ids, ora)
        print(f"[batch] {name} seq {b} (P={len(ps[b])}): {rep.summary()}", flush=True)
        assert rep.max_rel_err <= 2e-2
        assert rep.strict_ids, rep.summary()
