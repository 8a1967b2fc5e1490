"""Pins of the oracle's stored-weight products (oracle/matvec.c through
oracle/native.py), used for long full-size oracle runs.  CPU only.

What fixes them: exact integer arithmetic (small integers are exact in bf16,
float32 and float64, so every product and partial sum is exact and the result
must equal Python's integer dot product bit for bit), the float64 matrix
multiply of the widened weights (a library routine; only the order of the
additions differs, so agreement is to rounding), and whole oracle runs with and
without the stored-weight mapping."""

import numpy as np
import pytest

from oracle import DecoderOracle, dequantize_q8, quantize_q8
from oracle import native
from paper_2608_24204_amd import inputs
from tests.helpers import small_cfg

RNG = np.random.default_rng(4321)


def _bf16(f32):
    out = np.empty(f32.shape, np.uint16)
    inputs.f32_to_bf16_bits(np.ascontiguousarray(f32, np.float32), out)
    return out


@pytest.mark.parametrize("N,K,T", [(1, 1, 1), (3, 7, 1), (5, 8, 2), (9, 17, 3), (33, 1000, 1)])
def test_integer_products_are_exact(N, K, T):
    # |w| <= 64 and |x| <= 1000: products < 2^16, sums < 2^26, exact everywhere
    wi = RNG.integers(-64, 65, (N, K))
    xi = RNG.integers(-1000, 1001, (T, K))
    ref = np.array([[int(sum(int(a) * int(b) for a, b in zip(wi[n], xi[t]))) for n in range(N)]
                    for t in range(T)], dtype=np.float64)
    wf = wi.astype(np.float32)
    assert np.array_equal(native.matvec(_bf16(wf), xi.astype(np.float64)), ref)
    assert np.array_equal(native.matvec(wf, xi.astype(np.float64)), ref)


def test_non_square_orientation():
    # y = W x with W [N, K]: a transposed operand cannot even take these shapes,
    # and the value of each row is its own dot product
    W = np.arange(6, dtype=np.float32).reshape(2, 3)          # [[0,1,2],[3,4,5]]
    x = np.array([1.0, 10.0, 100.0])
    assert np.array_equal(native.matvec(W, x), np.array([210.0, 543.0]))
    with pytest.raises(ValueError):
        native.matvec(W, np.ones(2))


@pytest.mark.parametrize("N,K,T", [(64, 4099, 1), (257, 512, 3), (1000, 4096, 2)])
def test_matches_widened_matmul(N, K, T):
    f = RNG.standard_normal((N, K)).astype(np.float32) * np.float32(0.02)
    u = RNG.standard_normal((T, K))
    for w in (_bf16(f), f):
        ref = u @ native.widen(w).T
        got = native.matvec(w, u)
        assert np.max(np.abs(got - ref)) <= 1e-14 * np.max(np.abs(ref))


def test_widen_is_exact():
    f = RNG.standard_normal(1000).astype(np.float32)
    b = _bf16(f)
    w = native.widen(b)
    assert np.array_equal(w, inputs.bf16_bits_to_f32(b).astype(np.float64))
    assert np.array_equal(native.widen(f), f.astype(np.float64))


@pytest.mark.parametrize("wdt,tied", [("bf16", False), ("bf16", True), ("f32", False)])
def test_oracle_with_stored_weights_matches_plain(wdt, tied):
    cfg = small_cfg(weight_dtype=wdt, kv_dtype="bf16" if wdt == "bf16" else "f32",
                    tied_embeddings=tied, d_model=64, ffn_dim=96, vocab=300)
    w = inputs.make_weights(cfg, gain_std=0.1)
    prompt = inputs.make_prompt(cfg, 40)      # > C_MAX_ROWS rows: the widened route too
    a = DecoderOracle(cfg, inputs.weights_f64(cfg, w), max_seq=64)
    b = DecoderOracle(cfg, native.StoredWeights(w), max_seq=64)
    ia, la = a.generate(prompt, 8)
    ib, lb = b.generate(prompt, 8)
    assert ia == ib
    for x, y in zip(la, lb):
        assert np.max(np.abs(x - y)) <= 1e-12 * np.max(np.abs(x))


def test_oracle_with_quantised_store_matches_dequantised_f64():
    cfg = small_cfg(weight_dtype="bf16", kv_dtype="bf16", d_model=64, ffn_dim=96, vocab=300)
    w = inputs.make_weights(cfg, gain_std=0.1)
    f64, f32 = {}, {}
    for n, a in w.items():
        if a.ndim == 2:
            q, d = quantize_q8(inputs.bf16_bits_to_f32(a))
            f64[n] = dequantize_q8(q, d)
            f32[n] = f64[n].astype(np.float32)
            assert np.array_equal(f32[n].astype(np.float64), f64[n])    # q*d exact in fp32
        else:
            f64[n] = a.astype(np.float64)
            f32[n] = a
    prompt = inputs.make_prompt(cfg, 20)
    ia, la = DecoderOracle(cfg, f64, max_seq=40).generate(prompt, 6)
    ib, lb = DecoderOracle(cfg, native.StoredWeights(f32), max_seq=40).generate(prompt, 6)
    assert ia == ib
    for x, y in zip(la, lb):
        assert np.max(np.abs(x - y)) <= 1e-12 * np.max(np.abs(x))
