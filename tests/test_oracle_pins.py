"""Pins of the float64 oracle against things other than itself: closed forms,
invariants, brute force on tiny inputs, and library routines.  CPU only."""

import math

import numpy as np
import pytest
import torch

import oracle
from oracle import DecoderOracle
from paper_2608_24204_amd import configs, inputs
from tests.helpers import inf_rel, small_cfg

RNG = np.random.default_rng(1234)


def _oracle(cfg, gain_std=0.1, kv_round="none", seed=0, max_seq=None):
    w = inputs.weights_f64(cfg, inputs.make_weights(cfg, seed=seed, gain_std=gain_std))
    return DecoderOracle(cfg, w, kv_round=kv_round, max_seq=max_seq), w


# --------------------------------------------------------------------------- bf16
def test_bf16_round_matches_torch():
    # float32-representable inputs, so torch's float32 -> bf16 conversion (ties to
    # even) is a single rounding and must agree bit for bit
    x = RNG.standard_normal(200000).astype(np.float32) * np.float32(3.0)
    x[:8] = np.array([1 + 2**-8, 1 + 3 * 2**-8, -(1 + 2**-8), 2**-130, -2**-133 * 1.5,
                      3.38e38, 3.4e38, 0.0], np.float32)
    ours = oracle.bf16_round(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ours, ref)


# ------------------------------------------------------------------------ softmax
def test_softmax_rows_sum_to_one_and_shift_invariant():
    s = RNG.standard_normal((64, 37)) * 30
    p = oracle.softmax(s)
    assert np.max(np.abs(p.sum(-1) - 1)) <= 1e-14
    assert np.all(p >= 0)
    np.testing.assert_allclose(oracle.softmax(s + 123.25), p, rtol=1e-12, atol=1e-300)


# ---------------------------------------------------------------------- attention
def test_single_key_attention_returns_v():
    q = RNG.standard_normal((1, 4, 16))
    K = RNG.standard_normal((1, 2, 16))
    V = RNG.standard_normal((1, 2, 16))
    out = oracle.attend(q, K, V, np.array([0]), np.array([0]))
    for h in range(4):
        assert np.array_equal(out[0, h], V[0, h // 2])


def _attention_loops(q, K, V, q_pos, k_pos):
    T, Hq, hd = q.shape
    n, Hkv, _ = K.shape
    out = np.zeros_like(q)
    for t in range(T):
        for h in range(Hq):
            g = h * Hkv // Hq
            scores = []
            for j in range(n):
                if k_pos[j] <= q_pos[t]:
                    s = 0.0
                    for e in range(hd):
                        s += q[t, h, e] * K[j, g, e]
                    scores.append((j, s / math.sqrt(hd)))
            m = max(s for _, s in scores)
            z = sum(math.exp(s - m) for _, s in scores)
            for j, s in scores:
                w = math.exp(s - m) / z
                for e in range(hd):
                    out[t, h, e] += w * V[j, g, e]
    return out


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (4, 2), (6, 2), (5, 1)])
def test_attention_matches_triple_loop(Hq, Hkv):
    T, n, hd = 3, 7, 6
    q = RNG.standard_normal((T, Hq, hd))
    K = RNG.standard_normal((n, Hkv, hd))
    V = RNG.standard_normal((n, Hkv, hd))
    q_pos = np.arange(n - T, n)
    k_pos = np.arange(n)
    got = oracle.attend(q, K, V, q_pos, k_pos)
    ref = _attention_loops(q, K, V, q_pos, k_pos)
    assert np.max(np.abs(got - ref)) <= 1e-13


@pytest.mark.parametrize("Hq,Hkv", [(8, 2), (8, 8), (10, 2)])
def test_gqa_matches_library_attention_on_repeated_heads(Hq, Hkv):
    T, n, hd = 5, 19, 16
    q = RNG.standard_normal((T, Hq, hd))
    K = RNG.standard_normal((n, Hkv, hd))
    V = RNG.standard_normal((n, Hkv, hd))
    got = oracle.attend(q, K, V, np.arange(n - T, n), np.arange(n))
    # library: torch's attention in float64 on KV heads repeated per query group,
    # with an explicit boolean mask (queries are the last T positions)
    qt = torch.from_numpy(q).permute(1, 0, 2)                     # [Hq, T, hd]
    kt = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(Hq // Hkv, 0)
    vt = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(Hq // Hkv, 0)
    mask = torch.arange(n)[None, :] <= torch.arange(n - T, n)[:, None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask)
    assert np.max(np.abs(got - ref.permute(1, 0, 2).numpy())) <= 1e-12


# --------------------------------------------------------------------------- RoPE
def test_rope_properties():
    hd, base = 64, 500000.0
    z = RNG.standard_normal((40, 3, hd))
    pos = RNG.integers(0, 9000, 40)
    r = oracle.rope_rotate(z, pos, base)
    # norms of each rotated pair and of each head are preserved
    pn = z[..., :hd // 2] ** 2 + z[..., hd // 2:] ** 2
    rn = r[..., :hd // 2] ** 2 + r[..., hd // 2:] ** 2
    assert np.max(np.abs(pn - rn)) <= 1e-12
    # position 0 is the identity
    assert np.array_equal(oracle.rope_rotate(z, np.zeros(40, int), base), z)
    # pair 0 rotates by exactly the position (frequency 1): check against cos/sin
    p = 7
    one = np.zeros((1, 1, hd)); one[0, 0, 0] = 1.0
    rr = oracle.rope_rotate(one, np.array([p]), base)
    assert abs(rr[0, 0, 0] - math.cos(p)) < 1e-15 and abs(rr[0, 0, hd // 2] - math.sin(p)) < 1e-15
    # scores depend on relative position only
    q = RNG.standard_normal((1, 1, hd)); k = RNG.standard_normal((1, 1, hd))
    for m, n, s in [(5, 2, 100), (0, 0, 4000), (1000, 20, 3)]:
        a = np.sum(oracle.rope_rotate(q, [m], base) * oracle.rope_rotate(k, [n], base))
        b = np.sum(oracle.rope_rotate(q, [m + s], base) * oracle.rope_rotate(k, [n + s], base))
        assert abs(a - b) <= 1e-12 * max(1.0, abs(a))


# ------------------------------------------------------------------ RMSNorm/SiLU
def test_rmsnorm_closed_form():
    x = RNG.standard_normal((9, 33)) * 0.05
    eps = 1e-5
    y = oracle.rms_norm(x, np.ones(33), eps)
    ms = np.mean(x * x, -1)
    np.testing.assert_allclose(np.mean(y * y, -1), ms / (ms + eps), rtol=1e-13)
    g = RNG.standard_normal(33)
    np.testing.assert_allclose(oracle.rms_norm(x, g, eps), y * g, rtol=1e-14)
    # direction is kept: y is a positive multiple of x
    ratio = y / x
    assert np.all(ratio > 0) and np.max(np.abs(ratio - ratio[:, :1])) < 1e-12


def test_silu_values():
    assert oracle.silu(np.array([0.0]))[0] == 0.0
    assert abs(oracle.silu(np.array([40.0]))[0] - 40.0) < 1e-12
    assert abs(oracle.silu(np.array([-40.0]))[0]) < 1e-15
    z = np.array([1.0, -2.0, 0.5])
    np.testing.assert_allclose(oracle.silu(z), z * (1 / (1 + np.exp(-z))), rtol=1e-15)
    np.testing.assert_allclose(oracle.silu(np.array([1.0])), [0.7310585786300049], rtol=1e-15)


# ------------------------------------------------------------------------ argmax
def test_greedy_ties_and_last_index():
    v = np.zeros(1000); v[[17, 400, 999]] = 5.0
    assert oracle.greedy(v) == 17
    v = np.zeros(1000); v[-1] = 1e-300
    assert oracle.greedy(v) == 999
    with pytest.raises(FloatingPointError):
        oracle.greedy(np.array([0.0, np.nan]))


# -------------------------------------------------------------- whole forward
def _scalar_forward(cfg, w, tokens):
    """Scalar-loop forward over a whole sequence, written from the definition with
    Python floats only; returns logits of every position."""
    d, H, Hkv, hd, F = cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.ffn_dim
    T = len(tokens)

    def norm(vec, g):
        ms = sum(a * a for a in vec) / len(vec)
        r = 1.0 / math.sqrt(ms + cfg.rms_eps)
        return [a * r * gg for a, gg in zip(vec, g)]

    def matvec(W, vec):
        return [sum(W[i][j] * vec[j] for j in range(len(vec))) for i in range(len(W))]

    def rope(vec, p):
        out = list(vec)
        for j in range(hd // 2):
            th = p * cfg.rope_base ** (-2.0 * j / hd)
            a, b = vec[j], vec[j + hd // 2]
            out[j] = a * math.cos(th) - b * math.sin(th)
            out[j + hd // 2] = a * math.sin(th) + b * math.cos(th)
        return out

    xs = [list(w["tok_embeddings"][t]) for t in tokens]
    for l in range(cfg.n_layers):
        P = lambda n: w[f"layers.{l}.{n}"].tolist()
        Wq, Wk, Wv, Wo = P("wq"), P("wk"), P("wv"), P("wo")
        Wg, Wu, Wd = P("w_gate"), P("w_up"), P("w_down")
        ga, gf = P("attn_norm"), P("ffn_norm")
        Ks, Vs, Qs = [], [], []
        for i in range(T):
            u = norm(xs[i], ga)
            q, k, v = matvec(Wq, u), matvec(Wk, u), matvec(Wv, u)
            Qs.append([rope(q[h * hd:(h + 1) * hd], i) for h in range(H)])
            Ks.append([rope(k[g * hd:(g + 1) * hd], i) for g in range(Hkv)])
            Vs.append([v[g * hd:(g + 1) * hd] for g in range(Hkv)])
        new = []
        for i in range(T):
            att = []
            for h in range(H):
                g = h // (H // Hkv)
                sc = [sum(a * b for a, b in zip(Qs[i][h], Ks[j][g])) / math.sqrt(hd)
                      for j in range(i + 1)]
                m = max(sc)
                e = [math.exp(s - m) for s in sc]
                z = sum(e)
                att += [sum(e[j] / z * Vs[j][g][c] for j in range(i + 1)) for c in range(hd)]
            x = [a + b for a, b in zip(xs[i], matvec(Wo, att))]
            wn = norm(x, gf)
            gg, uu = matvec(Wg, wn), matvec(Wu, wn)
            hh = [a / (1 + math.exp(-a)) * b for a, b in zip(gg, uu)]
            new.append([a + b for a, b in zip(x, matvec(Wd, hh))])
        xs = new
    lm = (w["tok_embeddings"] if cfg.tied_embeddings else w["lm_head"]).tolist()
    return np.array([matvec(lm, norm(x, w["norm"].tolist())) for x in xs])


@pytest.mark.parametrize("tied,Hkv", [(False, 2), (True, 1)])
def test_forward_matches_scalar_loops(tied, Hkv):
    cfg = small_cfg(n_layers=2, d_model=12, n_heads=2, n_kv_heads=Hkv, head_dim=6,
                    ffn_dim=10, vocab=11, tied_embeddings=tied, key=51 + tied)
    orc, w = _oracle(cfg, gain_std=0.3)
    toks = [3, 7, 0, 10, 5]
    ref = _scalar_forward(cfg, w, toks)
    got = orc.full(toks)
    assert inf_rel(got, ref) <= 1e-12


def test_incremental_equals_recompute():
    cfg = small_cfg()
    orc, _ = _oracle(cfg)
    toks = inputs.make_prompt(cfg, 18)
    full = orc.full(toks)
    orc.reset()
    inc = [orc.prefill(toks[:7])]
    for t in toks[7:]:
        inc.append(orc.decode(int(t)))
    assert inf_rel(np.array(inc), full[6:]) <= 1e-12


def test_chunked_equals_oneshot_and_concat():
    cfg = small_cfg()
    orc, _ = _oracle(cfg)
    toks = inputs.make_prompt(cfg, 17)
    orc.reset(); one = orc.prefill(toks)
    orc.reset(); chunked = orc.prefill(toks, chunk=5)
    orc.reset(); orc.prefill(toks[:9]); cat = orc.prefill(toks[9:])
    assert inf_rel(chunked, one) <= 1e-12 and inf_rel(cat, one) <= 1e-12


def test_causality_future_tokens_do_not_change_past_logits():
    cfg = small_cfg()
    orc, _ = _oracle(cfg)
    toks = inputs.make_prompt(cfg, 12)
    a = orc.full(toks)
    toks2 = toks.copy(); toks2[8:] = (toks2[8:] + 5) % cfg.vocab
    b = orc.full(toks2)
    assert np.array_equal(a[:8], b[:8])
    assert not np.allclose(a[8:], b[8:])


def test_kv_round_stores_bf16_values():
    cfg = small_cfg(kv_dtype="bf16")
    orc, _ = _oracle(cfg, kv_round="bf16")
    orc.prefill(inputs.make_prompt(cfg, 6))
    K = orc.K[0][:6]
    assert np.array_equal(K, oracle.bf16_round(K))
    assert np.any(K != 0)


def test_generate_and_teacher_forcing_agree():
    cfg = small_cfg()
    orc, _ = _oracle(cfg)
    p = inputs.make_prompt(cfg)
    ids, logs = orc.generate(p, 5)
    assert len(ids) == 6 and all(oracle.greedy(l) == i for l, i in zip(logs, ids))
    tf = orc.teacher_forced(p, ids)
    for a, b in zip(tf, logs):
        assert np.array_equal(a, b)


def test_capacity_and_argument_errors():
    cfg = small_cfg()
    orc, _ = _oracle(cfg)
    with pytest.raises(ValueError):
        orc.prefill([])
    with pytest.raises(ValueError):
        orc.prefill([cfg.vocab])
    orc.reset()
    orc.prefill(np.zeros(cfg.max_seq, int))
    with pytest.raises(ValueError):
        orc.decode(0)


# ------------------------------------------------------ library cross-check (HF)
@pytest.mark.parametrize("tied,Hq,Hkv,base", [(False, 4, 2, 10000.0), (True, 6, 2, 500000.0),
                                             (False, 4, 4, 1e6)])
def test_matches_transformers_llama(tied, Hq, Hkv, base):
    transformers = pytest.importorskip("transformers")
    cfg = small_cfg(n_layers=3, d_model=48, n_heads=Hq, n_kv_heads=Hkv, head_dim=16,
                    ffn_dim=80, vocab=96, tied_embeddings=tied, rope_base=base, key=60)
    orc, w = _oracle(cfg, gain_std=0.2, max_seq=64)
    hf_cfg = transformers.LlamaConfig(
        vocab_size=cfg.vocab, hidden_size=cfg.d_model, intermediate_size=cfg.ffn_dim,
        num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
        num_key_value_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
        rms_norm_eps=cfg.rms_eps, rope_theta=cfg.rope_base,
        tie_word_embeddings=cfg.tied_embeddings, attention_bias=False, mlp_bias=False,
        hidden_act="silu", max_position_embeddings=256, torch_dtype="float64")
    hf_cfg.rope_parameters = {"rope_type": "default", "rope_theta": cfg.rope_base}
    model = transformers.LlamaForCausalLM(hf_cfg).to(torch.float64).eval()
    sd = {"model.embed_tokens.weight": w["tok_embeddings"], "model.norm.weight": w["norm"]}
    for l in range(cfg.n_layers):
        p, q = f"layers.{l}.", f"model.layers.{l}."
        sd.update({q + "input_layernorm.weight": w[p + "attn_norm"],
                   q + "self_attn.q_proj.weight": w[p + "wq"],
                   q + "self_attn.k_proj.weight": w[p + "wk"],
                   q + "self_attn.v_proj.weight": w[p + "wv"],
                   q + "self_attn.o_proj.weight": w[p + "wo"],
                   q + "post_attention_layernorm.weight": w[p + "ffn_norm"],
                   q + "mlp.gate_proj.weight": w[p + "w_gate"],
                   q + "mlp.up_proj.weight": w[p + "w_up"],
                   q + "mlp.down_proj.weight": w[p + "w_down"]})
    sd["lm_head.weight"] = w["tok_embeddings"] if tied else w["lm_head"]
    sd = {k: torch.from_numpy(np.ascontiguousarray(v)) for k, v in sd.items()}
    missing, unexpected = model.load_state_dict(sd, strict=False)
    assert not unexpected and all("rotary" in m for m in missing), (missing, unexpected)
    toks = inputs.make_prompt(cfg, 40)
    with torch.no_grad():
        ref = model(torch.from_numpy(toks.astype(np.int64))[None]).logits[0].numpy()
    got = orc.full(toks)
    # the library computes its norms and rotary angles in float32, so agreement is
    # at float32 level; a wrong convention (pairing, head map, transposed weight,
    # missing gain) differs at order one
    assert inf_rel(got, ref) <= 2e-5
    assert np.array_equal(got.argmax(-1), ref.argmax(-1))


# ------------------------------------------------------------- parameter counts
def test_parameter_counts_closed_form():
    c = configs.QWEN_32B
    per_layer = (40 * 128 + 2 * 8 * 128) * 5120 + 5120 * 40 * 128 + 3 * 27648 * 5120 + 2 * 5120
    total = 152064 * 5120 * 2 + 64 * per_layer + 5120
    assert c.n_params() == total
    assert abs(c.n_params() * 2 / 1e9 - 65.53) < 0.01       # ~65 GB in bf16
    assert configs.LLAMA_8B.n_params() == 8030261248          # Llama-3-8B shape
    assert configs.LLAMA_1B.n_params() == 1235814400          # Llama-3.2-1B shape (tied)
    for c in configs.CONFIGS.values():
        w = inputs.tensor_specs(c)
        assert sum(int(np.prod(s)) for _, s, _ in w) == c.n_params()
