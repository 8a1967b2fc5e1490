"""GPU parity: the HIP path (through the C ABI) against the float64 oracle on the
same seeded inputs.  Tolerances: logits max relative error (infinity norm) 1e-4
for fp32 weights, 2e-2 for bf16 weights; greedy ids identical at every step."""

from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2608_24204_amd import configs, inputs
from tests.parity import compare, oracle_run

pytestmark = pytest.mark.gpu

_W = {}


def weights_for(cfg, gain_std=0.0):
    key = (cfg, gain_std)
    if key not in _W:
        w = inputs.make_weights(cfg, gain_std=gain_std)
        _W.clear()  # keep at most one large weight set alive
        _W[key] = (w, inputs.weights_f64(cfg, w))
    return _W[key]


def make_model(cfg, w, **kw):
    from paper_2608_24204_amd.binding import WiciModel
    m = WiciModel(cfg, **kw)
    m.load_weights(w)
    return m


def tol_for(cfg):
    return 1e-4 if cfg.weight_dtype == "f32" else 2e-2


def run_parity(cfg, prompt, n_steps, gain_std=0.0, **kw):
    w, w64 = weights_for(cfg, gain_std)
    m = make_model(cfg, w, **kw)
    try:
        ids, logs = m.generate(prompt, n_steps, want_logits=True)
    finally:
        m.close()
    ora_ids, ora = oracle_run(cfg, w64, prompt, n_steps)
    rep = compare(ids, logs, ora_ids, ora)
    print(f"[parity] {cfg.name} P={len(prompt)} N={n_steps} {kw} -> {rep.summary()}", flush=True)
    return rep, ids, logs


# ---- small shapes exercising every kernel path --------------------------------------

SMALL = {
    "mha64_f32": configs.ModelConfig(name="t_mha64", key=70, n_layers=2, d_model=256, n_heads=4,
                                     n_kv_heads=4, head_dim=64, ffn_dim=512, vocab=1000,
                                     weight_dtype="f32", kv_dtype="f32", prompt_len=40,
                                     decode_steps=12),
    "gqa64_bf16": configs.ModelConfig(name="t_gqa64", key=71, n_layers=2, d_model=512, n_heads=8,
                                      n_kv_heads=2, head_dim=64, ffn_dim=1024, vocab=3001,
                                      prompt_len=77, decode_steps=12, tied_embeddings=True,
                                      rope_base=500000.0),
    "gqa128_bf16": configs.ModelConfig(name="t_gqa128", key=72, n_layers=2, d_model=512,
                                       n_heads=8, n_kv_heads=2, head_dim=128, ffn_dim=768,
                                       vocab=2500, prompt_len=150, decode_steps=12),
    "g5_bf16": configs.ModelConfig(name="t_g5", key=73, n_layers=1, d_model=640, n_heads=10,
                                   n_kv_heads=2, head_dim=128, ffn_dim=1536, vocab=1531,
                                   prompt_len=33, decode_steps=8, rope_base=1e6),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_small_configs_match_oracle(cuda_ok, name):
    cfg = SMALL[name]
    prompt = inputs.make_prompt(cfg)
    rep, _, _ = run_parity(cfg, prompt, cfg.decode_steps, gain_std=0.1, kv_page=16)
    assert rep.max_rel_err <= tol_for(cfg)
    assert rep.strict_ids, rep.summary()


def test_tiny_config(cuda_ok):
    cfg = configs.TINY
    rep, _, _ = run_parity(cfg, inputs.make_prompt(cfg), cfg.decode_steps)
    assert rep.max_rel_err <= 1e-4
    assert rep.strict_ids, rep.summary()


@pytest.mark.parametrize("P,chunk,page", [(1, 64, 16), (63, 64, 16), (65, 64, 32),
                                          (200, 64, 16), (129, 128, 128), (300, 2048, 64),
                                          (700, 2048, 64), (1000, 384, 16)])
def test_ragged_prompts_chunks_and_pages(cuda_ok, P, chunk, page):
    """From 8 key blocks of 64 the prefill attention splits the longest key walks
    in two and merges them: 700 positions in one chunk split query blocks 6..10
    (the last one ragged) and leave 0..5 whole; 1000 in chunks of 384 split
    every query block of the later chunks."""
    cfg = SMALL["gqa128_bf16"]
    prompt = inputs.make_prompt(cfg, P)
    rep, _, _ = run_parity(cfg, prompt, 20, gain_std=0.1, prefill_chunk=chunk, kv_page=page,
                           max_seq=P + 21)
    assert rep.max_rel_err <= 2e-2
    assert rep.strict_ids, rep.summary()


@pytest.mark.parametrize("P,max_seq,page", [(2030, 2048, 16), (2060, 2112, 16),
                                              (2100, 2200, 16), (2600, 4096, 64),
                                              (3000, 9000, 16), (5000, 16384, 128)])
def test_long_capacity_decode_attention(cuda_ok, P, max_seq, page):
    """The decode attention has one 64-position sub-chunk per 64 positions of
    capacity.  Up to 32 of them each is a split and the last split of a KV head
    to finish merges them in the same launch; beyond that each split walks
    ceil(sub-chunks / 32) consecutive sub-chunks under one online softmax (four
    teams of four wavefronts) and the same merge applies.  The cases give 32 and
    33 sub-chunks (either side of that switch), then 35 and 64 (two per split),
    141 (five: one team takes two) and 256 (eight, two per team), the most a
    launch accepts."""
    cfg = SMALL["gqa128_bf16"]
    prompt = inputs.make_prompt(cfg, P)
    rep, _, _ = run_parity(cfg, prompt, 12, gain_std=0.1, kv_page=page, max_seq=max_seq)
    assert rep.max_rel_err <= 2e-2
    assert rep.strict_ids, rep.summary()


@pytest.mark.parametrize("name,P,max_seq,page", [("gqa64_bf16", 2060, 2112, 16),
                                                   ("gqa64_bf16", 3000, 9000, 16),
                                                   ("mha64_f32", 2100, 2200, 16)])
def test_long_capacity_decode_attention_head_dim_64(cuda_ok, name, P, max_seq, page):
    """Past 32 sub-chunks at head dimension 64.  The bf16 cache runs on the
    matrix-core attention with splits of several sub-chunks (33 and 141
    sub-chunks); the fp32 cache on the vector kernel and the column-sliced merge
    kernel (35 splits)."""
    cfg = SMALL[name]
    prompt = inputs.make_prompt(cfg, P)
    rep, _, _ = run_parity(cfg, prompt, 12, gain_std=0.1, kv_page=page, max_seq=max_seq)
    assert rep.max_rel_err <= tol_for(cfg)
    assert rep.strict_ids, rep.summary()


@pytest.mark.parametrize("mode", ["bf16x3q", "bf16x3", "bf16x2", "bf16", "f32"])
def test_prefill_modes(cuda_ok, mode):
    cfg = SMALL["gqa64_bf16"]
    prompt = inputs.make_prompt(cfg, 130)
    rep, _, _ = run_parity(cfg, prompt, 4, gain_std=0.1, prefill_mode=mode, max_seq=140)
    assert rep.max_rel_err <= 2e-2
    if mode != "bf16":
        assert rep.max_rel_err <= 1e-3
        assert rep.strict_ids, rep.summary()


def _prefill_logits(cfg, w, prompt, n, **kw):
    m = make_model(cfg, w, max_seq=len(prompt) + n + 1, **kw)
    try:
        ids, logs = m.generate(prompt, n, want_logits=True)
    finally:
        m.close()
    return ids, np.stack(logs)


@pytest.mark.parametrize("planes,same_as", [((3, 2, 2, 2), "bf16x3q"), ((3, 2, 2, 2, 3), "bf16x3q"),
                                            ((3, 3, 3, 3), "bf16x3")])
def test_prefill_plane_fields_match_whole_modes(cuda_ok, planes, same_as):
    """Both modes store three bf16 terms; the per-product fields then choose
    exactly the terms each product of the whole mode reads, and the attention's
    query and probability terms (three when the field is left out), bit for bit."""
    cfg = SMALL["gqa128_bf16"]
    w, _ = weights_for(cfg, 0.1)
    prompt = inputs.make_prompt(cfg, 150)
    a = _prefill_logits(cfg, w, prompt, 3, prefill_mode="bf16x3", prefill_planes=planes)
    b = _prefill_logits(cfg, w, prompt, 3, prefill_mode=same_as)
    assert a[0] == b[0]
    assert np.array_equal(a[1], b[1])


def test_prefill_attention_with_two_terms(cuda_ok):
    """The attention field of prefill_planes: query and probabilities as two bf16
    terms (the default keeps three) against the oracle."""
    cfg = SMALL["gqa128_bf16"]
    prompt = inputs.make_prompt(cfg, 150)
    rep, _, _ = run_parity(cfg, prompt, 6, gain_std=0.1, prefill_mode="bf16x3",
                           prefill_planes=(3, 2, 2, 2, 2), max_seq=160)
    assert rep.max_rel_err <= 1e-3
    assert rep.strict_ids, rep.summary()


def test_kv_cache_holds_oracle_values(cuda_ok):
    cfg = SMALL["gqa128_bf16"]
    w, w64 = weights_for(cfg, 0.1)
    prompt = inputs.make_prompt(cfg, 70)
    m = make_model(cfg, w, kv_page=16, prefill_chunk=32, max_seq=80)
    try:
        tok, _ = m.prefill(prompt)
        m.decode_step(-1)
        kv = [m.read_kv(l, 0, 71) for l in range(cfg.n_layers)]
    finally:
        m.close()
    orc = oracle.DecoderOracle(cfg, w64, max_seq=80)
    otok = oracle.greedy(orc.prefill(prompt))
    assert otok == tok                 # same context for the decoded position
    orc.decode(otok)
    for l, (K, V) in enumerate(kv):
        for bits, o in ((K, orc.K[l][:71]), (V, orc.V[l][:71])):
            g = inputs.bf16_bits_to_f32(bits).astype(np.float64)
            assert np.array_equal(g, oracle.bf16_round(g))   # stored as bf16 values
            scale = np.max(np.abs(o))
            excess = float(np.max(np.abs(g - o) - np.abs(o) * 2.0 ** -7) / scale)
            print(f"[kv cache] layer {l}: differ {np.mean(g != o):.4f}, worst excess over one "
                  f"bf16 step {excess:.3g} of max|o|", flush=True)
            if l == 0:
                # layer 0 sees exact inputs: both sides round a value they computed
                # to bf16 and the GPU's value carries only float32 rounding, so the
                # results are at most one bf16 step apart (near zero: within the
                # float32 error of the value itself), and almost always identical
                bound = np.abs(o) * 2.0 ** -7 + scale * 2.0 ** -16
                viol = np.abs(g - o) > bound
                assert not viol.any(), (np.argwhere(viol)[:5], g[viol][:5], o[viol][:5])
                assert np.mean(g != o) < 0.01
            else:
                # deeper layers: the input already differs from the oracle's by the
                # float32 error of the layers below (and through attention by the
                # one-step storage differences of the cache below), a relative
                # error of order 2^-20 here.  Both sides then round to bf16, so
                # the results are at most one storage step apart plus that input
                # error; the bound allows 2^-14 of max|o| for it (measured worst:
                # 1.5e-6 = 2^-19.3 of max|o| beyond one step, on 0.46% of entries)
                bound = np.abs(o) * 2.0 ** -7 + scale * 2.0 ** -14
                viol = np.abs(g - o) > bound
                assert not viol.any(), (l, np.argwhere(viol)[:5], g[viol][:5], o[viol][:5])
                assert np.mean(g != o) < 0.02
                assert np.mean(g != o) < 0.2


def test_graph_replay_equals_eager_and_is_deterministic(cuda_ok):
    cfg = SMALL["gqa64_bf16"]
    w, _ = weights_for(cfg, 0.1)
    prompt = inputs.make_prompt(cfg, 50)
    out = []
    for graph in (True, False, True):
        m = make_model(cfg, w, graph=graph, max_seq=70)
        try:
            out.append(m.generate(prompt, 10, want_logits=True))
        finally:
            m.close()
    (i0, l0), (i1, l1), (i2, l2) = out
    assert i0 == i1 == i2
    for a, b, c in zip(l0, l1, l2):
        assert np.array_equal(a, b) and np.array_equal(a, c)


def test_split_prefill_equals_joint_prefill(cuda_ok):
    cfg = SMALL["gqa128_bf16"]
    w, _ = weights_for(cfg, 0.1)
    prompt = inputs.make_prompt(cfg, 90)
    m = make_model(cfg, w, max_seq=100)
    try:
        t_joint, l_joint = m.prefill(prompt, True)
        m.reset_kv()
        assert m.position == 0
        m.prefill(prompt[:37])
        t_split, l_split = m.prefill(prompt[37:], True)
        assert m.position == 90
    finally:
        m.close()
    assert t_joint == t_split
    assert np.max(np.abs(l_joint - l_split)) / np.max(np.abs(l_joint)) < 1e-4


@pytest.mark.parametrize("path", ["decode_step", "decode_n"])
def test_fault_drill_fails_the_decode_step(cuda_ok, path):
    """WICI_FLAG_FAULT_DRILL: the decode attention's merge in the last split block
    reports its splits as run on different XCDs, so the step fails with
    WICI_E_HIP and the model stays failed (the path a real misplacement takes;
    the kernels run normally).  Prefill has no in-launch merge and succeeds."""
    from paper_2608_24204_amd.binding import WICI_E_HIP, WICI_E_STATE, WiciError
    cfg = SMALL["gqa128_bf16"]
    w, _ = weights_for(cfg, 0.1)
    m = make_model(cfg, w, fault_drill=True)
    try:
        m.prefill(inputs.make_prompt(cfg, 40))
        with pytest.raises(WiciError) as e:
            m.decode_step() if path == "decode_step" else m.decode_n(4)
        assert e.value.status == WICI_E_HIP and "XCD" in str(e.value)
        with pytest.raises(WiciError) as e:
            m.decode_step()
        assert e.value.status == WICI_E_STATE
    finally:
        m.close()


def test_errors_and_state(cuda_ok):
    from paper_2608_24204_amd.binding import WiciError, WICI_E_ARG, WICI_E_CAPACITY, WICI_E_STATE
    cfg = SMALL["gqa64_bf16"]
    w, _ = weights_for(cfg, 0.1)
    m = make_model(cfg, w, max_seq=20)
    try:
        with pytest.raises(WiciError) as e:
            m.decode_step(-1)
        assert e.value.status == WICI_E_STATE
        with pytest.raises(WiciError) as e:
            m.prefill(np.zeros(21, np.int32))
        assert e.value.status == WICI_E_CAPACITY
        with pytest.raises(WiciError) as e:
            m.prefill([0, cfg.vocab])
        assert e.value.status == WICI_E_ARG
        assert m.position == 0
        m.prefill(np.arange(19) % cfg.vocab)
        tok, _ = m.decode_step(5)
        assert 0 <= tok < cfg.vocab and m.position == 20
        with pytest.raises(WiciError) as e:
            m.decode_step(-1)
        assert e.value.status == WICI_E_CAPACITY
        m.reset_kv()
        with pytest.raises(WiciError) as e:
            m.decode_step(-1)
        assert e.value.status == WICI_E_STATE
        t2, _ = m.prefill(np.arange(19) % cfg.vocab)
        assert 0 <= t2 < cfg.vocab
    finally:
        m.close()


def test_non_finite_logits_are_reported(cuda_ok):
    from paper_2608_24204_amd.binding import WiciError, WICI_E_NUMERIC, WICI_E_STATE
    cfg = SMALL["mha64_f32"]
    w, _ = weights_for(cfg, 0.1)
    w = dict(w)
    lm = w["lm_head"].copy()
    lm[17, 3] = np.nan
    w["lm_head"] = lm
    m = make_model(cfg, w, max_seq=20)
    try:
        with pytest.raises(WiciError) as e:
            m.prefill([1, 2, 3])
        assert e.value.status == WICI_E_NUMERIC
        with pytest.raises(WiciError) as e:
            m.decode_step(-1)          # no token to feed back
        assert e.value.status == WICI_E_STATE
        with pytest.raises(WiciError) as e:
            m.decode_step(4)           # an explicit token runs, and fails again
        assert e.value.status == WICI_E_NUMERIC
    finally:
        m.close()
